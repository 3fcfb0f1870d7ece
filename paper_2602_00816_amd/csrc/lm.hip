// Transformer kernels for the two gradient passes, run in lockstep.
//
// Every activation is carried as a pair of fp32 tensors: m = (x+ + x-)/2 and
// d = (x+ - x-)/2, where x+ and x- are the activation at theta + eps v and at
// theta - eps v.  The bilinear contractions run on MFMA (gemm.hip); every
// other operation here reconstructs the two points x+- = m +- d in fp64,
// evaluates the operation at each point in fp64, and stores the mean and half
// difference of the two results.  The half difference therefore keeps full
// relative precision however small the step eps is.
#include "kernels.h"

namespace fdh {

namespace {

constexpr int NT = 256;

unsigned grid_for(int64_t n) {
  int64_t g = (n + NT - 1) / NT;
  if (g > 262144) g = 262144;
  if (g < 1) g = 1;
  return (unsigned)g;
}

#define GRID_LOOP(i, n) for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < (n); i += (int64_t)gridDim.x * blockDim.x)

template <typename T>
__device__ inline void put_pair(PairT<T> o, int64_t i, double p, double q) {
  stf(o.m, i, (float)(0.5 * (p + q)));
  stf(o.d, i, (float)(0.5 * (p - q)));
}

template <typename T>
__global__ void cast_pair_kernel(PairT<T> o, const float* m, const float* d, int64_t n) {
  GRID_LOOP(i, n) {
    stf(o.m, i, m[i]);
    stf(o.d, i, d[i]);
  }
}

// ---- embedding ----------------------------------------------------------------
// token ids outside [0, V) are clamped so that no access leaves the tables;
// the embedding forward reports them (bad_tok[0] = 1) and the call that
// launched it turns that into an invalid-argument error
__device__ inline int clamp_tok(int t, int V) { return t < 0 ? 0 : (t >= V ? V - 1 : t); }

template <typename T>
__global__ void embed_fwd_kernel(PairF x, const int32_t* tok, int T_, int S, int dm, int V, const T* the, const float* ve,
                                 const T* thp, const float* vp, double eps, int* bad_tok) {
  const int64_t n = (int64_t)T_ * dm;
  GRID_LOOP(i, n) {
    const int t = (int)(i / dm), j = (int)(i % dm);
    const int tk = tok[t];
    if ((tk < 0 || tk >= V) && bad_tok && j == 0) bad_tok[0] = 1;
    const int64_t r = (int64_t)clamp_tok(tk, V) * dm + j;
    double xp = (double)ldf(the, r) + eps * (double)ve[r];
    double xm = (double)ldf(the, r) - eps * (double)ve[r];
    if (thp) {
      const int64_t pr = (int64_t)(t % S) * dm + j;
      xp += (double)ldf(thp, pr) + eps * (double)vp[pr];
      xm += (double)ldf(thp, pr) - eps * (double)vp[pr];
    }
    x.m[i] = (float)(0.5 * (xp + xm));
    x.d[i] = (float)(0.5 * (xp - xm));
  }
}

// ---- LayerNorm / RMSNorm ---------------------------------------------------------
// one workgroup per row
template <typename T>
__global__ __launch_bounds__(NT) void norm_fwd_kernel(PairT<T> y, const float* xm, const float* xd, int dm, bool ln,
                                                      const T* thg, const float* vg, const T* thb, const float* vb,
                                                      double eps, double neps) {
  __shared__ double sh[NT / 64];
  const int64_t row = blockIdx.x;
  const float* rm = xm + row * dm;
  const float* rd = xd + row * dm;
  double mup = 0.0, mum = 0.0;
  if (ln) {
    double sp = 0.0, sm = 0.0;
    for (int j = threadIdx.x; j < dm; j += NT) {
      sp += (double)rm[j] + (double)rd[j];
      sm += (double)rm[j] - (double)rd[j];
    }
    mup = block_sum<NT>(sp, sh) / dm;
    mum = block_sum<NT>(sm, sh) / dm;
  }
  double qp = 0.0, qm = 0.0;
  for (int j = threadIdx.x; j < dm; j += NT) {
    const double a = (double)rm[j] + (double)rd[j] - mup;
    const double b = (double)rm[j] - (double)rd[j] - mum;
    qp += a * a;
    qm += b * b;
  }
  const double rp = 1.0 / sqrt(block_sum<NT>(qp, sh) / dm + neps);
  const double rmi = 1.0 / sqrt(block_sum<NT>(qm, sh) / dm + neps);
  for (int j = threadIdx.x; j < dm; j += NT) {
    const double g = ldf(thg, j), dg = eps * (double)vg[j];
    double op = ((double)rm[j] + (double)rd[j] - mup) * rp * (g + dg);
    double om = ((double)rm[j] - (double)rd[j] - mum) * rmi * (g - dg);
    if (thb) {
      const double b = ldf(thb, j), db = eps * (double)vb[j];
      op += b + db;
      om += b - db;
    }
    put_pair(y, row * dm + j, op, om);
  }
}

// NORM_BWD_ROWS consecutive rows per workgroup.  Besides dx (and its operand-type
// copy), each workgroup adds up the gain-gradient terms of its rows per column
// in fp64, in row order (and dy.d for the LayerNorm bias), and writes one
// partial row; a column sum over the workgroups finishes the gradient.  A
// column's sum lives in LDS and is only ever touched by the thread that owns
// the column, so no barrier guards it.
template <typename T>
__global__ __launch_bounds__(NT) void norm_bwd_kernel(PairF dx, PairT<T> dxo, const float* dresm, const float* dresd,
                                                      const float* xm, const float* xd, const float* dym,
                                                      const float* dyd, int rows, int dm, bool ln, const T* thg,
                                                      const float* vg, double eps, double neps, double* gpart,
                                                      double* bpart) {
  extern __shared__ double cacc[];  // [dm] gain partials, then [dm] bias partials
  __shared__ double sh[NT / 64];
  for (int j = threadIdx.x; j < dm; j += NT) {
    cacc[j] = 0.0;
    if (bpart) cacc[dm + j] = 0.0;
  }
  const int r0 = blockIdx.x * NORM_BWD_ROWS, r1 = min(rows, r0 + NORM_BWD_ROWS);
  for (int row = r0; row < r1; ++row) {
    const int64_t o = (int64_t)row * dm;
    double mup = 0.0, mum = 0.0;
    if (ln) {
      double sp = 0.0, sm = 0.0;
      for (int j = threadIdx.x; j < dm; j += NT) {
        sp += (double)xm[o + j] + (double)xd[o + j];
        sm += (double)xm[o + j] - (double)xd[o + j];
      }
      mup = block_sum<NT>(sp, sh) / dm;
      mum = block_sum<NT>(sm, sh) / dm;
    }
    double qp = 0.0, qm = 0.0;
    for (int j = threadIdx.x; j < dm; j += NT) {
      const double a = (double)xm[o + j] + (double)xd[o + j] - mup;
      const double b = (double)xm[o + j] - (double)xd[o + j] - mum;
      qp += a * a;
      qm += b * b;
    }
    const double rp = 1.0 / sqrt(block_sum<NT>(qp, sh) / dm + neps);
    const double rmi = 1.0 / sqrt(block_sum<NT>(qm, sh) / dm + neps);
    // means of dxhat and dxhat * xhat at both points
    double s1p = 0.0, s1m = 0.0, s2p = 0.0, s2m = 0.0;
    for (int j = threadIdx.x; j < dm; j += NT) {
      const double g = ldf(thg, j), dg = eps * (double)vg[j];
      const double xhp = ((double)xm[o + j] + (double)xd[o + j] - mup) * rp;
      const double xhm = ((double)xm[o + j] - (double)xd[o + j] - mum) * rmi;
      const double dhp = ((double)dym[o + j] + (double)dyd[o + j]) * (g + dg);
      const double dhm = ((double)dym[o + j] - (double)dyd[o + j]) * (g - dg);
      s1p += dhp;
      s1m += dhm;
      s2p += dhp * xhp;
      s2m += dhm * xhm;
    }
    const double a1p = ln ? block_sum<NT>(s1p, sh) / dm : 0.0;
    const double a1m = ln ? block_sum<NT>(s1m, sh) / dm : 0.0;
    const double a2p = block_sum<NT>(s2p, sh) / dm;
    const double a2m = block_sum<NT>(s2m, sh) / dm;
    for (int j = threadIdx.x; j < dm; j += NT) {
      const double g = ldf(thg, j), dg = eps * (double)vg[j];
      const double xhp = ((double)xm[o + j] + (double)xd[o + j] - mup) * rp;
      const double xhm = ((double)xm[o + j] - (double)xd[o + j] - mum) * rmi;
      const double dyp = (double)dym[o + j] + (double)dyd[o + j];
      const double dymi = (double)dym[o + j] - (double)dyd[o + j];
      const double dhp = dyp * (g + dg), dhm = dymi * (g - dg);
      const double dxp = rp * (dhp - a1p - xhp * a2p);
      const double dxm = rmi * (dhm - a1m - xhm * a2m);
      const double rm0 = dresm ? (double)dresm[o + j] : 0.0;
      const double rd0 = dresd ? (double)dresd[o + j] : 0.0;
      const float om = (float)(rm0 + 0.5 * (dxp + dxm)), od = (float)(rd0 + 0.5 * (dxp - dxm));
      dx.m[o + j] = om;
      dx.d[o + j] = od;
      if (dxo.m) {
        stf(dxo.m, o + j, om);
        stf(dxo.d, o + j, od);
      }
      cacc[j] += 0.5 * (dyp * xhp - dymi * xhm);
      if (bpart) cacc[dm + j] += (double)dyd[o + j];
    }
  }
  for (int j = threadIdx.x; j < dm; j += NT) {
    gpart[(int64_t)blockIdx.x * dm + j] = cacc[j];
    if (bpart) bpart[(int64_t)blockIdx.x * dm + j] = cacc[dm + j];
  }
}

// Same computation with one wavefront per row (rows of 256 CPL columns): lane
// l holds the float4 chunks at columns 256 c + 4 l.  The row reductions are
// wavefront sums (no barriers); each pass rereads its operands, which after
// the first pass come from the caches.  Each wavefront adds the
// gain and bias terms of its rows per column in LDS (fp32, at most
// NORM_BWD_ROWS / 4 rows), and the four wavefronts' sums are added in fp64 in
// wavefront order.
template <typename T>
__device__ inline float4 ld4f(const T* p, int64_t i) {
  if constexpr (sizeof(T) == 4) {
    return *reinterpret_cast<const float4*>(p + i);
  } else {
    const uint2 u = *reinterpret_cast<const uint2*>(p + i);
    return make_float4(bf16_to_f32((bf16_t)(u.x & 0xFFFF)), bf16_to_f32((bf16_t)(u.x >> 16)),
                       bf16_to_f32((bf16_t)(u.y & 0xFFFF)), bf16_to_f32((bf16_t)(u.y >> 16)));
  }
}
template <typename T>
__device__ inline void st4f(T* p, int64_t i, float a, float b, float c, float d) {
  if constexpr (sizeof(T) == 4) {
    *reinterpret_cast<float4*>(p + i) = make_float4(a, b, c, d);
  } else {
    *reinterpret_cast<uint2*>(p + i) = make_uint2((uint32_t)f32_to_bf16(a) | ((uint32_t)f32_to_bf16(b) << 16),
                                                  (uint32_t)f32_to_bf16(c) | ((uint32_t)f32_to_bf16(d) << 16));
  }
}
__device__ inline float f4e(const float4& v, int e) { return e == 0 ? v.x : (e == 1 ? v.y : (e == 2 ? v.z : v.w)); }

// Norm forward with one wavefront per row (rows of 256 CPL columns, lane l
// at columns 256 c + 4 l), NORM_FWD_ROWS rows per workgroup: wavefront
// reductions, x reread from the caches between the passes.  Same arithmetic
// as norm_fwd_kernel.
constexpr int NORM_FWD_ROWS = 4;
// An empty statement that claims to modify the cached row values, so that the
// compiler recomputes their fp64 conversions in each pass instead of keeping
// them live (twice the registers) from the previous one.  No instruction.
template <int CPL>
__device__ inline void reload_barrier(float4 (&a)[CPL], float4 (&b)[CPL]) {
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    asm volatile("" : "+v"(a[c].x), "+v"(a[c].y), "+v"(a[c].z), "+v"(a[c].w));
    asm volatile("" : "+v"(b[c].x), "+v"(b[c].y), "+v"(b[c].z), "+v"(b[c].w));
  }
}

template <typename T, int CPL>
__global__ __launch_bounds__(NT) void norm_fwd_wave_kernel(PairT<T> y, const float* xm, const float* xd, int rows, bool ln,
                                                           const T* thg, const float* vg, const T* thb, const float* vb,
                                                           double eps, double neps) {
  constexpr int DM = 256 * CPL;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  auto ld = [](const float* p, int64_t i) { return *reinterpret_cast<const float4*>(p + i); };
  const int r0 = blockIdx.x * NORM_FWD_ROWS;
  for (int i = wave; i < NORM_FWD_ROWS; i += 4) {
    const int row = r0 + i;
    if (row >= rows) break;
    const int64_t o = (int64_t)row * DM + 4 * lane;
    // the lane's 4 CPL elements of both channels, loaded once (all loads in flight together)
    float4 xa[CPL], xb[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      xa[c] = ld(xm, o + 256 * c);
      xb[c] = ld(xd, o + 256 * c);
    }
    double mup = 0.0, mum = 0.0;
    if (ln) {
      double sp = 0.0, sm = 0.0;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const float4 a = xa[c], b = xb[c];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          sp += (double)f4e(a, e) + (double)f4e(b, e);
          sm += (double)f4e(a, e) - (double)f4e(b, e);
        }
      }
      mup = wave_sum(sp) / DM;
      mum = wave_sum(sm) / DM;
    }
    // keep the fp32 values, not their fp64 conversions, live across the passes
    reload_barrier<CPL>(xa, xb);
    double qp = 0.0, qm = 0.0;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const float4 a = xa[c], b = xb[c];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double p = (double)f4e(a, e) + (double)f4e(b, e) - mup;
        const double q = (double)f4e(a, e) - (double)f4e(b, e) - mum;
        qp += p * p;
        qm += q * q;
      }
    }
    const double rp = 1.0 / sqrt(wave_sum(qp) / DM + neps);
    const double rmi = 1.0 / sqrt(wave_sum(qm) / DM + neps);
    reload_barrier<CPL>(xa, xb);
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const int col = 256 * c + 4 * lane;
      const float4 a = xa[c], b = xb[c];
      const float4 g4 = ld4f(thg, col), v4 = ld(vg, col);
      float4 b4 = make_float4(0.f, 0.f, 0.f, 0.f), w4 = b4;
      if (thb) {
        b4 = ld4f(thb, col);
        w4 = ld(vb, col);
      }
      float om[4], od[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double g = f4e(g4, e), dg = eps * (double)f4e(v4, e);
        double op = ((double)f4e(a, e) + (double)f4e(b, e) - mup) * rp * (g + dg);
        double on = ((double)f4e(a, e) - (double)f4e(b, e) - mum) * rmi * (g - dg);
        if (thb) {
          const double bb = f4e(b4, e), db = eps * (double)f4e(w4, e);
          op += bb + db;
          on += bb - db;
        }
        om[e] = (float)(0.5 * (op + on));
        od[e] = (float)(0.5 * (op - on));
      }
      st4f(y.m, o + 256 * c, om[0], om[1], om[2], om[3]);
      st4f(y.d, o + 256 * c, od[0], od[1], od[2], od[3]);
    }
  }
}

template <typename T, int CPL>
__global__ __launch_bounds__(NT) void norm_bwd_wave_kernel(PairF dx, PairT<T> dxo, const float* dresm, const float* dresd,
                                                           const float* xm, const float* xd, const float* dym,
                                                           const float* dyd, int rows, bool ln, const T* thg,
                                                           const float* vg, double eps, double neps, double* gpart,
                                                           double* bpart) {
  constexpr int DM = 256 * CPL;
  // per-wavefront column sums (gain, bias); a lane only touches its own columns
  __shared__ float cg[4][DM], cb[4][DM];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int c = 0; c < CPL; ++c) {
    *reinterpret_cast<float4*>(&cg[wave][256 * c + 4 * lane]) = make_float4(0.f, 0.f, 0.f, 0.f);
    *reinterpret_cast<float4*>(&cb[wave][256 * c + 4 * lane]) = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  auto ld = [](const float* p, int64_t i) { return *reinterpret_cast<const float4*>(p + i); };
  const int r0 = blockIdx.x * NORM_BWD_ROWS;
  for (int i = wave; i < NORM_BWD_ROWS; i += 4) {
    const int row = r0 + i;
    if (row >= rows) break;
    const int64_t o = (int64_t)row * DM + 4 * lane;
    double mup = 0.0, mum = 0.0;
    float4 xac[CPL], xbc[CPL];   // the row of x, kept in registers for the later passes
    if (ln) {
      double sp = 0.0, sm = 0.0;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const float4 xa = ld(xm, o + 256 * c), xb = ld(xd, o + 256 * c);
        xac[c] = xa;
        xbc[c] = xb;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          sp += (double)f4e(xa, e) + (double)f4e(xb, e);
          sm += (double)f4e(xa, e) - (double)f4e(xb, e);
        }
      }
      mup = wave_sum(sp) / DM;
      mum = wave_sum(sm) / DM;
    }
    double rp, rmi, a1p = 0.0, a1m = 0.0, a2p, a2m;
    if (!ln) {
      // RMSNorm (no mean): sum x^2 and sum dxhat * x in one pass over x and
      // dy; mean(dxhat * xhat) = r * mean(dxhat * x)
      double qp = 0.0, qm = 0.0, tp = 0.0, tm = 0.0;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const int col = 256 * c + 4 * lane;
        const float4 xa = ld(xm, o + 256 * c), xb = ld(xd, o + 256 * c);
        xac[c] = xa;
        xbc[c] = xb;
        const float4 ya = ld(dym, o + 256 * c), yb = ld(dyd, o + 256 * c);
        const float4 g4 = ld4f(thg, col), v4 = ld(vg, col);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const double g = f4e(g4, e), dg = eps * (double)f4e(v4, e);
          const double p = (double)f4e(xa, e) + (double)f4e(xb, e);
          const double q = (double)f4e(xa, e) - (double)f4e(xb, e);
          qp += p * p;
          qm += q * q;
          tp += ((double)f4e(ya, e) + (double)f4e(yb, e)) * (g + dg) * p;
          tm += ((double)f4e(ya, e) - (double)f4e(yb, e)) * (g - dg) * q;
        }
      }
      rp = 1.0 / sqrt(wave_sum(qp) / DM + neps);
      rmi = 1.0 / sqrt(wave_sum(qm) / DM + neps);
      a2p = rp * (wave_sum(tp) / DM);
      a2m = rmi * (wave_sum(tm) / DM);
    } else {
      // LayerNorm: the variance, sum dxhat and sum dxhat * (x - mu) in one
      // pass over dy, x from the registers; mean(dxhat * xhat) =
      // r * mean(dxhat * (x - mu))
      double qp = 0.0, qm = 0.0, s1p = 0.0, s1m = 0.0, tp = 0.0, tm = 0.0;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const int col = 256 * c + 4 * lane;
        const float4 xa = xac[c], xb = xbc[c];
        const float4 ya = ld(dym, o + 256 * c), yb = ld(dyd, o + 256 * c);
        const float4 g4 = ld4f(thg, col), v4 = ld(vg, col);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const double g = f4e(g4, e), dg = eps * (double)f4e(v4, e);
          const double p = (double)f4e(xa, e) + (double)f4e(xb, e) - mup;
          const double q = (double)f4e(xa, e) - (double)f4e(xb, e) - mum;
          const double dhp = ((double)f4e(ya, e) + (double)f4e(yb, e)) * (g + dg);
          const double dhm = ((double)f4e(ya, e) - (double)f4e(yb, e)) * (g - dg);
          qp += p * p;
          qm += q * q;
          s1p += dhp;
          s1m += dhm;
          tp += dhp * p;
          tm += dhm * q;
        }
      }
      rp = 1.0 / sqrt(wave_sum(qp) / DM + neps);
      rmi = 1.0 / sqrt(wave_sum(qm) / DM + neps);
      a1p = wave_sum(s1p) / DM;
      a1m = wave_sum(s1m) / DM;
      a2p = rp * (wave_sum(tp) / DM);
      a2m = rmi * (wave_sum(tm) / DM);
    }
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const int col = 256 * c + 4 * lane;
      const float4 xa = xac[c], xb = xbc[c];
      const float4 ya = ld(dym, o + 256 * c), yb = ld(dyd, o + 256 * c);
      const float4 g4 = ld4f(thg, col), v4 = ld(vg, col);
      const float4 ra = dresm ? ld(dresm, o + 256 * c) : make_float4(0.f, 0.f, 0.f, 0.f);
      const float4 rb = dresd ? ld(dresd, o + 256 * c) : make_float4(0.f, 0.f, 0.f, 0.f);
      float om[4], od[4], tg[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double g = f4e(g4, e), dg = eps * (double)f4e(v4, e);
        const double xhp = ((double)f4e(xa, e) + (double)f4e(xb, e) - mup) * rp;
        const double xhm = ((double)f4e(xa, e) - (double)f4e(xb, e) - mum) * rmi;
        const double dyp = (double)f4e(ya, e) + (double)f4e(yb, e);
        const double dymi = (double)f4e(ya, e) - (double)f4e(yb, e);
        const double dhp = dyp * (g + dg), dhm = dymi * (g - dg);
        const double dxp = rp * (dhp - a1p - xhp * a2p);
        const double dxm = rmi * (dhm - a1m - xhm * a2m);
        om[e] = (float)((double)f4e(ra, e) + 0.5 * (dxp + dxm));
        od[e] = (float)((double)f4e(rb, e) + 0.5 * (dxp - dxm));
        tg[e] = (float)(0.5 * (dyp * xhp - dymi * xhm));
      }
      *reinterpret_cast<float4*>(dx.m + o + 256 * c) = make_float4(om[0], om[1], om[2], om[3]);
      *reinterpret_cast<float4*>(dx.d + o + 256 * c) = make_float4(od[0], od[1], od[2], od[3]);
      if (dxo.m) {
        st4f(dxo.m, o + 256 * c, om[0], om[1], om[2], om[3]);
        st4f(dxo.d, o + 256 * c, od[0], od[1], od[2], od[3]);
      }
      float4* pg = reinterpret_cast<float4*>(&cg[wave][col]);
      float4* pb = reinterpret_cast<float4*>(&cb[wave][col]);
      const float4 g0 = *pg, b0 = *pb;
      *pg = make_float4(g0.x + tg[0], g0.y + tg[1], g0.z + tg[2], g0.w + tg[3]);
      *pb = make_float4(b0.x + yb.x, b0.y + yb.y, b0.z + yb.z, b0.w + yb.w);
    }
  }
  // the four wavefronts' column sums, added in fp64 in wavefront order
  __syncthreads();
  for (int j = threadIdx.x; j < DM; j += NT) {
    gpart[(int64_t)blockIdx.x * DM + j] = (double)cg[0][j] + (double)cg[1][j] + (double)cg[2][j] + (double)cg[3][j];
    if (bpart)
      bpart[(int64_t)blockIdx.x * DM + j] = (double)cb[0][j] + (double)cb[1][j] + (double)cb[2][j] + (double)cb[3][j];
  }
}

// ---- column sums ---------------------------------------------------------------
constexpr int COLSUM_CHUNKS = 64;
__global__ void colsum_stage1(double* partial, const float* X, int rows, int C, int64_t ld) {
  const int j = blockIdx.x * NT + threadIdx.x;
  if (j >= C) return;
  const int c = blockIdx.y;
  const int per = (rows + COLSUM_CHUNKS - 1) / COLSUM_CHUNKS;
  const int r0 = c * per, r1 = min(rows, r0 + per);
  double s = 0.0;
  for (int r = r0; r < r1; ++r) s += (double)X[(int64_t)r * ld + j];
  partial[(int64_t)c * C + j] = s;
}
__global__ void colsum64_stage1(double* partial, const double* X, int rows, int C) {
  const int j = blockIdx.x * NT + threadIdx.x;
  if (j >= C) return;
  const int c = blockIdx.y;
  const int per = (rows + COLSUM_CHUNKS - 1) / COLSUM_CHUNKS;
  const int r0 = c * per, r1 = min(rows, r0 + per);
  double s = 0.0;
  for (int r = r0; r < r1; ++r) s += X[(int64_t)r * C + j];
  partial[(int64_t)c * C + j] = s;
}
__global__ void colsum_stage2(float* out, const double* partial, int C, double scale, bool acc) {
  const int j = blockIdx.x * NT + threadIdx.x;
  if (j >= C) return;
  double s = 0.0;
  for (int c = 0; c < COLSUM_CHUNKS; ++c) s += partial[(int64_t)c * C + j];
  s *= scale;
  out[j] = acc ? (float)((double)out[j] + s) : (float)s;
}

// ---- RoPE ----------------------------------------------------------------------
__global__ void rope_table_kernel(double* cs, int S, int dh, double base) {
  const int half = dh / 2;
  GRID_LOOP(i, (int64_t)S * half) {
    const int s = (int)(i / half), f = (int)(i % half);
    const double inv = pow(base, -(double)(2 * f) / (double)dh);
    const double ang = (double)s * inv;
    cs[(int64_t)s * dh + 2 * f] = cos(ang);
    cs[(int64_t)s * dh + 2 * f + 1] = sin(ang);
  }
}

// Both channels in one pass.  A thread takes 4 consecutive columns f0..f0+3
// of the first half of a q or k head together with their rotate-half
// partners f0+dh/2.., reads each once and writes both rotated quadruples
// (packed); v columns (and q/k without RoPE) are cast 4 at a time.
template <typename T, typename TI>
__global__ void qkv_rope_kernel(PairT<T> out, const TI* inm, const TI* ind, int S, int ncols, int nqk, int dh,
                                const double* cs, bool rope, bool inverse, bool copy_v) {
  const int t = blockIdx.y;
  const int u = blockIdx.x * blockDim.x + threadIdx.x;
  const int half = dh / 2, qpu = half / 4;      // units per q/k head
  const int qu = rope ? nqk * qpu : 0;          // rotated units
  const int vu = copy_v ? (ncols - (rope ? nqk * dh : 0)) / 4 : 0;
  const int64_t o = (int64_t)t * ncols;
  if (u < qu) {
    const int head = u / qpu, f0 = 4 * (u % qpu);
    const int c = head * dh + f0;
    const double* row = cs + (int64_t)(t % S) * dh;
    double co[4], si[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      co[e] = row[2 * (f0 + e)];
      si[e] = inverse ? -row[2 * (f0 + e) + 1] : row[2 * (f0 + e) + 1];
    }
    const TI* ins[2] = {inm, ind};
    T* outs[2] = {out.m, out.d};
#pragma unroll
    for (int ch = 0; ch < 2; ++ch) {
      // (in place when ins == outs: this thread alone reads and writes these 8 elements)
      const float4 x = ld4f(ins[ch], o + c);
      const float4 y = ld4f(ins[ch], o + c + half);
      float lo[4], hi[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double xe = f4e(x, e), ye = f4e(y, e);
        lo[e] = (float)(xe * co[e] - ye * si[e]);
        hi[e] = (float)(ye * co[e] + xe * si[e]);
      }
      st4f(outs[ch], o + c, lo[0], lo[1], lo[2], lo[3]);
      st4f(outs[ch], o + c + half, hi[0], hi[1], hi[2], hi[3]);
    }
  } else if (u < qu + vu) {
    const int c = (rope ? nqk * dh : 0) + 4 * (u - qu);
    const float4 a = ld4f(inm, o + c), b = ld4f(ind, o + c);
    st4f(out.m, o + c, a.x, a.y, a.z, a.w);
    st4f(out.d, o + c, b.x, b.y, b.z, b.w);
  }
}

// ---- causal softmax and its backward, both points ---------------------------------------
constexpr int MAXE = 16;  // row elements per thread (rows up to 4096)

template <typename T>
__global__ __launch_bounds__(NT) void attn_softmax_kernel(PairT<T> P, const float* Sm, const float* Sd, int S) {
  __shared__ double sh[NT / 64];
  const int64_t r = blockIdx.x;
  const int i = (int)(r % S);
  const int64_t base = r * (int64_t)S;
  const int len = i + 1;
  double ep[MAXE], em[MAXE];
  double mx = -1e300;
#pragma unroll
  for (int e = 0; e < MAXE; ++e) {
    const int j = threadIdx.x + e * NT;
    if (j < len) mx = fmax(mx, (double)Sm[base + j]);
  }
  mx = block_max<NT>(mx, sh);
  double zp = 0.0, zm = 0.0;
#pragma unroll
  for (int e = 0; e < MAXE; ++e) {
    const int j = threadIdx.x + e * NT;
    ep[e] = em[e] = 0.0;
    if (j < len) {
      const double a = (double)Sm[base + j] - mx, b = (double)Sd[base + j];
      ep[e] = exp(a + b);
      em[e] = exp(a - b);
      zp += ep[e];
      zm += em[e];
    }
  }
  zp = block_sum<NT>(zp, sh);
  zm = block_sum<NT>(zm, sh);
  const double izp = 1.0 / zp, izm = 1.0 / zm;
#pragma unroll
  for (int e = 0; e < MAXE; ++e) {
    const int j = threadIdx.x + e * NT;
    if (j < S) put_pair(P, base + j, ep[e] * izp, em[e] * izm);
  }
}

template <typename T>
__global__ __launch_bounds__(NT) void attn_dsoftmax_kernel(PairT<T> dS, const T* Pm, const T* Pd, const float* dPm,
                                                           const float* dPd, int S) {
  __shared__ double sh[NT / 64];
  const int64_t r = blockIdx.x;
  const int i = (int)(r % S);
  const int64_t base = r * (int64_t)S;
  const int len = i + 1;
  double dp = 0.0, dm = 0.0;
#pragma unroll
  for (int e = 0; e < MAXE; ++e) {
    const int j = threadIdx.x + e * NT;
    if (j < len) {
      const double pm = ldf(Pm, base + j), pd = ldf(Pd, base + j);
      const double gm = dPm[base + j], gd = dPd[base + j];
      dp += (pm + pd) * (gm + gd);
      dm += (pm - pd) * (gm - gd);
    }
  }
  dp = block_sum<NT>(dp, sh);
  dm = block_sum<NT>(dm, sh);
#pragma unroll
  for (int e = 0; e < MAXE; ++e) {
    const int j = threadIdx.x + e * NT;
    if (j < S) {
      double sp = 0.0, sn = 0.0;
      if (j < len) {
        const double pm = ldf(Pm, base + j), pd = ldf(Pd, base + j);
        const double gm = dPm[base + j], gd = dPd[base + j];
        sp = (pm + pd) * (gm + gd - dp);
        sn = (pm - pd) * (gm - gd - dm);
      }
      put_pair(dS, base + j, sp, sn);
    }
  }
}

// Wavefront-per-row versions (4 rows per workgroup).  Row i of a causal score
// matrix has i+1 live entries; entries i < j < roundup(i+1, 256) are written
// as zeros, because the MFMA tiles that contract over a row read exactly up
// to that boundary; entries beyond it are never read and not written.
// The softmax at both points uses exp(Sm - c +- Sd) = exp(Sm - c) (cosh Sd +- sinh Sd):
// per live entry a = exp(Sm - c) cosh(Sd) and b = exp(Sm - c) sinh(Sd), both
// with full relative precision however small Sd is, so that e+- = a +- b and
//   P.m = (a Zm - b Zd) / (Z+ Z-),  P.d = (b Zm - a Zd) / (Z+ Z-),
// with Zm = sum a and Zd = sum b (fp64 sums) the mean and half difference of
// Z+- = sum e+-.  exp(Sm - c) is formed in fp32: its rounding is common to the
// two points.
__device__ inline int zero_end(int i, int S) { return min(S, ((i + 256) / 256) * 256); }

template <typename T, int PER>
__global__ __launch_bounds__(256) void attn_softmax_w(PairT<T> P, const float* Sm, const float* Sd, int nrows, int S) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= nrows) return;
  const int i = (int)(r % S);
  const int64_t base = r * (int64_t)S;
  const int len = i + 1;
  float av[PER], bv[PER];
  float mx = -3.0e38f;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int j = lane + 64 * e;
    av[e] = (j < len) ? Sm[base + j] : -3.0e38f;
    bv[e] = (j < len) ? Sd[base + j] : 0.f;
    mx = fmaxf(mx, av[e]);
  }
  mx = wave_max(mx);
  double Zm = 0.0, Zd = 0.0;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int j = lane + 64 * e;
    if (j < len) {
      const float ea = expf(av[e] - mx);
      const float b = bv[e];
      av[e] = ea * coshf(b);
      bv[e] = ea * sinhf(b);
      Zm += (double)av[e];
      Zd += (double)bv[e];
    } else {
      av[e] = bv[e] = 0.f;
    }
  }
  Zm = wave_sum(Zm);
  Zd = wave_sum(Zd);
  const double inv = 1.0 / ((Zm + Zd) * (Zm - Zd));
  const int ze = zero_end(i, S);
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int j = lane + 64 * e;
    if (j < ze) {
      const double a = av[e], b = bv[e];
      stf(P.m, base + j, (float)((a * Zm - b * Zd) * inv));
      stf(P.d, base + j, (float)((b * Zm - a * Zd) * inv));
    }
  }
}

template <typename T, int PER>
__global__ __launch_bounds__(256) void attn_dsoftmax_w(PairT<T> dS, const T* Pm, const T* Pd, const float* dPm,
                                                       const float* dPd, int nrows, int S) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= nrows) return;
  const int i = (int)(r % S);
  const int64_t base = r * (int64_t)S;
  const int len = i + 1;
  double dp = 0.0, dm = 0.0;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int j = lane + 64 * e;
    if (j < len) {
      const double pm = ldf(Pm, base + j), pd = ldf(Pd, base + j);
      const double gm = dPm[base + j], gd = dPd[base + j];
      dp += (pm + pd) * (gm + gd);
      dm += (pm - pd) * (gm - gd);
    }
  }
  dp = wave_sum(dp);
  dm = wave_sum(dm);
  const int ze = zero_end(i, S);
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int j = lane + 64 * e;
    if (j < ze) {
      double sp = 0.0, sn = 0.0;
      if (j < len) {
        const double pm = ldf(Pm, base + j), pd = ldf(Pd, base + j);
        const double gm = dPm[base + j], gd = dPd[base + j];
        sp = (pm + pd) * (gm + gd - dp);
        sn = (pm - pd) * (gm - gd - dm);
      }
      put_pair(dS, base + j, sp, sn);
    }
  }
}

__global__ void group_sum_kernel(float* out, int64_t out_ld, const float* in, int T_, int Hk, int G, int dh) {
  const int64_t n = (int64_t)T_ * Hk * dh;
  GRID_LOOP(i, n) {
    const int t = (int)(i / (Hk * dh)), c = (int)(i % (Hk * dh));
    const int kh = c / dh, e = c % dh;
    double s = 0.0;
    for (int g = 0; g < G; ++g) s += in[(int64_t)t * (Hk * G * dh) + (int64_t)(kh * G + g) * dh + e];
    out[(int64_t)t * out_ld + c] = (float)s;
  }
}

// ---- activations ------------------------------------------------------------------
__device__ inline double gelu_t(double u) {
  const double k = 0.7978845608028654, a = 0.044715;
  return 0.5 * u * (1.0 + tanh(k * (u + a * u * u * u)));
}
__device__ inline double gelu_t_grad(double u) {
  const double k = 0.7978845608028654, a = 0.044715;
  const double t = tanh(k * (u + a * u * u * u));
  return 0.5 * (1.0 + t) + 0.5 * u * (1.0 - t * t) * k * (1.0 + 3.0 * a * u * u);
}
__device__ inline double sigm(double x) { return 1.0 / (1.0 + exp(-x)); }

// SwiGLU output at both points, (s(a) v_a, s(b) v_b) with s(x) = x sigmoid(x),
// gate a, b = gm +- gd and up u = um +- ud, returned as its half sum om and half
// difference od, in fp32 without forming the two values and subtracting them:
//   (s(a) + s(b)) / 2 is taken directly;
//   (s(a) - s(b)) / 2 = (gd (sig(a) + sig(b)) + gm (sig(a) - sig(b))) / 2, and
//   sig(a) - sig(b) = sig(a) sig(-b) (1 - e^(-2 gd)) with expm1 for the last
//   factor, so the difference channel keeps fp32 relative accuracy for any gd
//   (no loss of order gd / gm);
//   om = S um + D ud and od = S ud + D um for the gate's half sum S and half
//   difference D.
__device__ inline void swiglu_pair(float gm, float gd, float um, float ud, float& om, float& od) {
  const float a = gm + gd, b = gm - gd;
  const float eb = expf(-b);
  const float sa = 1.f / (1.f + expf(-a)), sb = 1.f / (1.f + eb);
  const float snb = b < 0.f ? 1.f - sb : eb * sb;   // sig(-b), accurate on both sides
  const float dsig = sa * snb * -expm1f(-2.f * gd);
  const float S = 0.5f * (a * sa + b * sb), D = 0.5f * (gd * (sa + sb) + gm * dsig);
  om = S * um + D * ud;
  od = S * ud + D * um;
}

// SwiGLU backward at both points in the same channel form: for the upstream
// gradient z = zm +- zd, the gate gradient z v s'(g) and the up gradient
// z s(g), with s'(x) = sig(x) (1 + x sig(-x)).  Every factor is split into its
// half sum and half difference and a product of two split factors is formed as
// (xm ym + xd yd, xm yd + xd ym), which is exact before rounding.  The half
// difference of s' is (sig(a) - sig(b) + h(a) - h(b)) / 2 with
// h(x) = x sig'(x), sig' = sig(x) sig(-x), and
//   h(a) - h(b) = gd (sig'(a) + sig'(b)) + gm (sig'(a) - sig'(b)),
//   sig'(a) - sig'(b) = (sig(a) - sig(b)) (1 - sig(a) - sig(b)),
// so no term subtracts two values of the full size of s'.
__device__ inline void swiglu_bwd_pair(float gm, float gd, float um, float ud, float zm, float zd, float& am,
                                       float& ad, float& bm, float& bd) {
  const float a = gm + gd, b = gm - gd;
  const float ea = expf(-a), eb = expf(-b);
  const float sa = 1.f / (1.f + ea), sb = 1.f / (1.f + eb);
  const float sna = a < 0.f ? 1.f - sa : ea * sa, snb = b < 0.f ? 1.f - sb : eb * sb;
  const float dsig = sa * snb * -expm1f(-2.f * gd);
  const float pa = sa * sna, pb = sb * snb;   // sig'(a), sig'(b)
  const float S1 = 0.5f * (sa * (1.f + a * sna) + sb * (1.f + b * snb));
  const float D1 = 0.5f * (dsig + gd * (pa + pb) + gm * dsig * (1.f - sa - sb));
  const float S0 = 0.5f * (a * sa + b * sb), D0 = 0.5f * (gd * (sa + sb) + gm * dsig);
  const float xm = zm * um + zd * ud, xd = zm * ud + zd * um;   // z v
  am = xm * S1 + xd * D1;
  ad = xm * D1 + xd * S1;
  bm = zm * S0 + zd * D0;
  bd = zm * D0 + zd * S0;
}

template <typename T>
__global__ void gelu_fwd_kernel(PairT<T> z, const T* um, const T* ud, int64_t n) {
  GRID_LOOP(i, n) {
    const double a = ldf(um, i), b = ldf(ud, i);
    const double up = a + b, un = a - b;
    put_pair(z, i, gelu_t(up), gelu_t(un));
  }
}
template <typename T>
__global__ void gelu_bwd_kernel(PairT<T> du, float* dudf, const T* um, const T* ud, const float* dzm,
                                const float* dzd, int64_t n) {
  GRID_LOOP(i, n) {
    const double a = ldf(um, i), b = ldf(ud, i);
    const double up = a + b, un = a - b;
    const double gp = ((double)dzm[i] + (double)dzd[i]) * gelu_t_grad(up);
    const double gn = ((double)dzm[i] - (double)dzd[i]) * gelu_t_grad(un);
    put_pair(du, i, gp, gn);
    if (dudf) dudf[i] = (float)(0.5 * (gp - gn));
  }
}
// Vectorised forms: grid.y = row, each thread 4 consecutive columns of the
// F gate (and F up) columns; F % 4 == 0.  Same arithmetic as the scalar forms.
template <typename T>
__global__ void swiglu_fwd4_kernel(PairT<T> z, const T* gum, const T* gud, int F) {
  const int c = 4 * (blockIdx.x * blockDim.x + threadIdx.x);
  if (c >= F) return;
  const int64_t t = blockIdx.y;
  const int64_t ig = t * 2 * F + c, iu = ig + F, io = t * F + c;
  const float4 gm = ld4f(gum, ig), gd = ld4f(gud, ig);
  const float4 um = ld4f(gum, iu), ud = ld4f(gud, iu);
  float om[4], od[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) swiglu_pair(f4e(gm, e), f4e(gd, e), f4e(um, e), f4e(ud, e), om[e], od[e]);
  st4f(z.m, io, om[0], om[1], om[2], om[3]);
  st4f(z.d, io, od[0], od[1], od[2], od[3]);
}
template <typename T>
__global__ void swiglu_bwd4_kernel(PairT<T> dgu, const T* gum, const T* gud, const float* dzm, const float* dzd,
                                   int F) {
  const int c = 4 * (blockIdx.x * blockDim.x + threadIdx.x);
  if (c >= F) return;
  const int64_t t = blockIdx.y;
  const int64_t ig = t * 2 * F + c, iu = ig + F, io = t * F + c;
  const float4 gm = ld4f(gum, ig), gd = ld4f(gud, ig);
  const float4 um = ld4f(gum, iu), ud = ld4f(gud, iu);
  const float4 zm = *reinterpret_cast<const float4*>(dzm + io), zd = *reinterpret_cast<const float4*>(dzd + io);
  float am[4], ad[4], bm[4], bd[4];
#pragma unroll
  for (int e = 0; e < 4; ++e)
    swiglu_bwd_pair(f4e(gm, e), f4e(gd, e), f4e(um, e), f4e(ud, e), f4e(zm, e), f4e(zd, e), am[e], ad[e], bm[e], bd[e]);
  st4f(dgu.m, ig, am[0], am[1], am[2], am[3]);
  st4f(dgu.d, ig, ad[0], ad[1], ad[2], ad[3]);
  st4f(dgu.m, iu, bm[0], bm[1], bm[2], bm[3]);
  st4f(dgu.d, iu, bd[0], bd[1], bd[2], bd[3]);
}

template <typename T>
__global__ void swiglu_fwd_kernel(PairT<T> z, const T* gum, const T* gud, int rows, int F) {
  const int64_t n = (int64_t)rows * F;
  GRID_LOOP(i, n) {
    const int64_t t = i / F, c = i % F;
    const int64_t ig = t * 2 * F + c, iu = ig + F;
    float om, od;
    swiglu_pair(ldf(gum, ig), ldf(gud, ig), ldf(gum, iu), ldf(gud, iu), om, od);
    stf(z.m, i, om);
    stf(z.d, i, od);
  }
}
template <typename T>
__global__ void swiglu_bwd_kernel(PairT<T> dgu, const T* gum, const T* gud, const float* dzm, const float* dzd,
                                  int rows, int F) {
  const int64_t n = (int64_t)rows * F;
  GRID_LOOP(i, n) {
    const int64_t t = i / F, c = i % F;
    const int64_t ig = t * 2 * F + c, iu = ig + F;
    float am, ad, bm, bd;
    swiglu_bwd_pair(ldf(gum, ig), ldf(gud, ig), ldf(gum, iu), ldf(gud, iu), dzm[i], dzd[i], am, ad, bm, bd);
    stf(dgu.m, ig, am);
    stf(dgu.d, ig, ad);
    stf(dgu.m, iu, bm);
    stf(dgu.d, iu, bd);
  }
}

// ---- cross-entropy, both points -------------------------------------------------------------
// The logits of position t predict the label of position t + 1: the next token,
// or lab[t + 1] when labels are given; a label of IGNORE_LABEL (padding,
// masked prompt) leaves the row out.  inv_n scales every kept row.
// e^b and e^-b as c + s and c - s with c = cosh b and s = sinh b: for
// |b| < 1/16 their Taylor series to b^8 and b^9 (the first omitted terms are
// below 2^-40 / 10! of the sum), otherwise from exp.
__device__ inline void exp_pm(double b, double& ep, double& en) {
  if (fabs(b) < 0.0625) {
    const double b2 = b * b;
    const double c = 1.0 + b2 * (1.0 / 2 + b2 * (1.0 / 24 + b2 * (1.0 / 720 + b2 * (1.0 / 40320))));
    const double sn = b * (1.0 + b2 * (1.0 / 6 + b2 * (1.0 / 120 + b2 * (1.0 / 5040 + b2 * (1.0 / 362880)))));
    ep = c + sn;
    en = c - sn;
  } else {
    ep = exp(b);
    en = exp(-b);
  }
}

template <typename T>
__global__ __launch_bounds__(NT) void ce_kernel(PairT<T> dl, double* rowloss, const float* lm, const float* ld,
                                                const int32_t* tok, const int32_t* lab, int T_, int S, int V,
                                                double inv_n) {
  __shared__ double sh[NT / 64];
  const int64_t t = blockIdx.x;
  const int64_t o = t * (int64_t)V;
  const bool last = (t % S) == (S - 1);
  const int raw = last ? IGNORE_LABEL : (lab ? lab[t + 1] : tok[t + 1]);
  if (raw == IGNORE_LABEL) {
    for (int j = threadIdx.x; j < V; j += NT) put_pair(dl, o + j, 0.0, 0.0);
    if (threadIdx.x == 0) { rowloss[t] = 0.0; rowloss[T_ + t] = 0.0; }
    return;
  }
  const int y = clamp_tok(raw, V);
  // exp(a +- b) = E e^+-b with E = exp(a) shared by both points.  For bf16
  // models E is taken in fp32 (a common factor of the two channels, so its
  // rounding never cancels in their half difference) and e^+-b from exp_pm;
  // fp32 models keep both exponentials in fp64.
  auto both = [&](double a, double b, double& xp, double& xn) {
    if constexpr (sizeof(T) == 2) {
      const double E = (double)__expf((float)a);
      double ep, en;
      exp_pm(b, ep, en);
      xp = E * ep;
      xn = E * en;
    } else {
      xp = exp(a + b);
      xn = exp(a - b);
    }
  };
  // one pass for the row maximum and the sums: each thread keeps its sums
  // relative to its own running maximum mt, rescaled by exp(old mt - new mt)
  // when mt rises, then relative to the row maximum mx.  The rescale factors
  // are common to both points (taken in fp32 for bf16 models, like E).
  auto rescale = [&](double d) {
    if constexpr (sizeof(T) == 2) return (double)__expf((float)d);
    else return exp(d);
  };
  double mt = -1e300, zp = 0.0, zm = 0.0;
  for (int j = threadIdx.x; j < V; j += NT) {
    const double av = (double)lm[o + j], b = (double)ld[o + j];
    if (av > mt) {
      const double f = mt > -1e300 ? rescale(mt - av) : 0.0;
      zp *= f;
      zm *= f;
      mt = av;
    }
    double xp, xn;
    both(av - mt, b, xp, xn);
    zp += xp;
    zm += xn;
  }
  const double mx = block_max<NT>(mt, sh);
  const double fr = mt > -1e300 ? rescale(mt - mx) : 0.0;
  zp = block_sum<NT>(zp * fr, sh);
  zm = block_sum<NT>(zm * fr, sh);
  const double izp = 1.0 / zp, izm = 1.0 / zm;
  for (int j = threadIdx.x; j < V; j += NT) {
    const double a = (double)lm[o + j] - mx, b = (double)ld[o + j];
    double xp, xn;
    both(a, b, xp, xn);
    double pp = xp * izp, pn = xn * izm;
    if (j == y) { pp -= 1.0; pn -= 1.0; }
    put_pair(dl, o + j, pp * inv_n, pn * inv_n);
  }
  if (threadIdx.x == 0) {
    const double a = (double)lm[o + y] - mx, b = (double)ld[o + y];
    rowloss[t] = (log(zp) - (a + b)) * inv_n;
    rowloss[T_ + t] = (log(zm) - (a - b)) * inv_n;
  }
}

__global__ void loss_sum_kernel(double* out2, const double* rowloss, int T_, bool acc) {
  __shared__ double sh[NT / 64];
  double a = 0.0, b = 0.0;
  // fixed assignment of rows to threads, fixed reduction tree
  for (int t = threadIdx.x; t < T_; t += NT) { a += rowloss[t]; b += rowloss[T_ + t]; }
  a = block_sum<NT>(a, sh);
  b = block_sum<NT>(b, sh);
  if (threadIdx.x == 0) {
    out2[0] = acc ? out2[0] + a : a;
    out2[1] = acc ? out2[1] + b : b;
  }
}

// out[0] += number of targets of one [B, S] batch (positions t % S < S - 1
// whose label at t + 1 is not IGNORE_LABEL; all of them without labels),
// out[1] += number of labels outside [0, V) other than IGNORE_LABEL,
// out[2] += number of tokens outside [0, V).
__global__ void count_targets_kernel(int64_t* out, const int32_t* tok, const int32_t* lab, int B, int S, int V) {
  __shared__ double sh[NT / 64];
  const int64_t n = (int64_t)B * S;
  double c = 0.0, bad = 0.0, badt = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += NT) {
    const int x = tok[i];
    if (x < 0 || x >= V) badt += 1.0;
    const int64_t t = i % S;
    if (t == S - 1) continue;
    const int y = lab ? lab[i + 1] : 0;
    if (y == IGNORE_LABEL) continue;
    if (y < 0 || y >= V) bad += 1.0;
    else c += 1.0;
  }
  // counts below 2^53 are exact in fp64
  c = block_sum<NT>(c, sh);
  bad = block_sum<NT>(bad, sh);
  badt = block_sum<NT>(badt, sh);
  if (threadIdx.x == 0) {
    out[0] += (int64_t)c;
    out[1] += (int64_t)bad;
    out[2] += (int64_t)badt;
  }
}

// ---- embedding backward --------------------------------------------------------------
constexpr int SORT_N = 16384;  // keys = token << 14 | position, positions < 2^14
__global__ __launch_bounds__(1024) void token_sort_kernel(uint32_t* keys, const int32_t* tok, int T_, int V) {
  __shared__ uint32_t k[SORT_N];
  int n2 = 1;
  while (n2 < T_) n2 <<= 1;
  for (int i = threadIdx.x; i < n2; i += 1024)
    k[i] = (i < T_) ? (((uint32_t)clamp_tok(tok[i], V) << 14) | (uint32_t)i) : 0xFFFFFFFFu;
  __syncthreads();
  for (int size = 2; size <= n2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = threadIdx.x; i < n2; i += 1024) {
        const int p = i ^ stride;
        if (p > i) {
          const bool up = (i & size) == 0;
          const uint32_t a = k[i], b = k[p];
          if ((a > b) == up) { k[i] = b; k[p] = a; }
        }
      }
      __syncthreads();
    }
  }
  for (int i = threadIdx.x; i < T_; i += 1024) keys[i] = k[i];
}

// One workgroup per (sorted position, NT-column chunk); only segment starts
// work.  The segment end is found by binary search in the sorted keys, and
// the segment's rows are summed with 8 partial sums (row q of the segment
// into partial q % 8, combined in a fixed order), so that frequent tokens
// (hundreds of rows under a Zipf distribution) keep 8 loads in flight.
__global__ void embed_bwd_kernel(float* hv, const uint32_t* keys, const float* dxd, int T_, int dm, double inv_eps,
                                 bool acc) {
  const int j = blockIdx.x;
  const uint32_t tk = keys[j] >> 14;
  if (j > 0 && (keys[j - 1] >> 14) == tk) return;
  int lo = j + 1, hi = T_;   // first position with a larger token
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if ((keys[mid] >> 14) == tk) lo = mid + 1;
    else hi = mid;
  }
  const int e = lo;
  const int c = blockIdx.y * NT + threadIdx.x;
  if (c >= dm) return;
  double s[8] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
  int q = j;
  for (; q + 8 <= e; q += 8) {
#pragma unroll
    for (int u = 0; u < 8; ++u) s[u] += (double)dxd[(int64_t)(keys[q + u] & 0x3FFFu) * dm + c];
  }
  for (int u = 0; q < e; ++q, ++u) s[u] += (double)dxd[(int64_t)(keys[q] & 0x3FFFu) * dm + c];
  const double t = ((s[0] + s[1]) + (s[2] + s[3])) + ((s[4] + s[5]) + (s[6] + s[7]));
  const int64_t idx = (int64_t)tk * dm + c;
  hv[idx] = acc ? (float)((double)hv[idx] + t * inv_eps) : (float)(t * inv_eps);
}

__global__ void pos_bwd_kernel(float* hv, const float* dxd, int B, int S, int dm, double inv_eps, bool acc) {
  const int64_t n = (int64_t)S * dm;
  GRID_LOOP(i, n) {
    const int s = (int)(i / dm), c = (int)(i % dm);
    double a = 0.0;
    for (int b = 0; b < B; ++b) a += (double)dxd[((int64_t)b * S + s) * dm + c];
    const float x = (float)(a * inv_eps);
    hv[i] = acc ? hv[i] + x : x;
  }
}

}  // namespace

// ================================ launchers ==============================================
template <typename T>
hipError_t launch_cast_pair(PairT<T> out, const float* m, const float* d, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(cast_pair_kernel<T>, dim3(grid_for(n)), dim3(NT), 0, s, out, m, d, n);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_embed_fwd(PairF x, const int32_t* tok, int T_, int S, int dm, int V, const T* the, const float* ve,
                            const T* thp, const float* vp, double eps, int* bad_tok, hipStream_t s) {
  hipLaunchKernelGGL(embed_fwd_kernel<T>, dim3(grid_for((int64_t)T_ * dm)), dim3(NT), 0, s, x, tok, T_, S, dm, V, the,
                     ve, thp, vp, eps, bad_tok);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_norm_fwd(PairT<T> y, const float* xm, const float* xd, int rows, int dm, bool ln, const T* thg,
                           const float* vg, const T* thb, const float* vb, double eps, float neps, hipStream_t s) {
  const dim3 g(ceil_div(rows, NORM_FWD_ROWS));
#define NFW(C) hipLaunchKernelGGL((norm_fwd_wave_kernel<T, C>), g, dim3(NT), 0, s, y, xm, xd, rows, ln, thg, vg, thb, vb, eps, \
                                  (double)neps)
  if (dm == 512) NFW(2);
  else if (dm == 1024) NFW(4);
  else if (dm == 2048) NFW(8);
  else hipLaunchKernelGGL(norm_fwd_kernel<T>, dim3(rows), dim3(NT), 0, s, y, xm, xd, dm, ln, thg, vg, thb, vb, eps, (double)neps);
#undef NFW
  return hipGetLastError();
}

template <typename T>
hipError_t launch_norm_bwd(PairF dx, PairT<T> dxo, const float* dresm, const float* dresd, const float* xm, const float* xd,
                           const float* dym, const float* dyd, int rows, int dm, bool ln, const T* thg,
                           const float* vg, double eps, float neps, double* gpart, double* bpart, hipStream_t s) {
  const dim3 g(norm_bwd_groups(rows));
  // one wavefront per row where the row is 512, 1024 or 2048 columns
#define NBW(C) hipLaunchKernelGGL((norm_bwd_wave_kernel<T, C>), g, dim3(NT), 0, s, dx, dxo, dresm, dresd, xm, xd, dym, dyd, \
                                  rows, ln, thg, vg, eps, (double)neps, gpart, bpart)
  if (dm == 512) NBW(2);
  else if (dm == 1024) NBW(4);
  else if (dm == 2048) NBW(8);
  else {
    const size_t lds = (size_t)dm * (bpart ? 2 : 1) * sizeof(double);
    if (lds > 64 * 1024) return hipErrorInvalidValue;
    hipLaunchKernelGGL(norm_bwd_kernel<T>, g, dim3(NT), lds, s, dx, dxo, dresm, dresd, xm, xd, dym, dyd, rows, dm, ln, thg,
                       vg, eps, (double)neps, gpart, bpart);
  }
#undef NBW
  return hipGetLastError();
}

hipError_t launch_colsum(float* out, const float* X, int rows, int C, int64_t ld, double scale, bool acc, double* partial,
                         hipStream_t s) {
  hipLaunchKernelGGL(colsum_stage1, dim3(ceil_div(C, NT), COLSUM_CHUNKS), dim3(NT), 0, s, partial, X, rows, C, ld);
  hipLaunchKernelGGL(colsum_stage2, dim3(ceil_div(C, NT)), dim3(NT), 0, s, out, (const double*)partial, C, scale, acc);
  return hipGetLastError();
}

hipError_t launch_colsum_f64(float* out, const double* X, int rows, int C, double scale, bool acc, double* partial,
                             hipStream_t s) {
  hipLaunchKernelGGL(colsum64_stage1, dim3(ceil_div(C, NT), COLSUM_CHUNKS), dim3(NT), 0, s, partial, X, rows, C);
  hipLaunchKernelGGL(colsum_stage2, dim3(ceil_div(C, NT)), dim3(NT), 0, s, out, (const double*)partial, C, scale, acc);
  return hipGetLastError();
}

hipError_t launch_rope_table(double* cs, int S, int dh, double base, hipStream_t s) {
  hipLaunchKernelGGL(rope_table_kernel, dim3(grid_for((int64_t)S * dh / 2)), dim3(NT), 0, s, cs, S, dh, base);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_rope_inplace(PairT<T> qkv, int T_, int S, int Hq, int Hk, int dh, const double* cs, hipStream_t s) {
  const int ncols = (Hq + 2 * Hk) * dh;
  const int units = (Hq + Hk) * dh / 8;
  const dim3 g(ceil_div(units, NT), T_);
  hipLaunchKernelGGL((qkv_rope_kernel<T, T>), g, dim3(NT), 0, s, qkv, (const T*)qkv.m, (const T*)qkv.d, S, ncols, Hq + Hk, dh,
                     cs, true, false, false);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_qkv_bwd_post(PairT<T> out, float* gm, float* gd, int T_, int S, int Hq, int Hk, int dh,
                               const double* cs, bool rope, hipStream_t s) {
  const int ncols = (Hq + 2 * Hk) * dh;
  const int units = (rope ? (Hq + Hk) * dh / 8 : 0) + (ncols - (rope ? (Hq + Hk) * dh : 0)) / 4;
  const dim3 g(ceil_div(units, NT), T_);
  hipLaunchKernelGGL((qkv_rope_kernel<T, float>), g, dim3(NT), 0, s, out, (const float*)gm, (const float*)gd, S, ncols,
                     Hq + Hk, dh, cs, rope, true, true);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_attn_softmax(PairT<T> P, const float* Sm, const float* Sd, int nrows, int S, hipStream_t s) {
  if (S > 4096) return hipErrorInvalidValue;
  const dim3 g(ceil_div(nrows, 4)), b(256);
  if (S <= 512) hipLaunchKernelGGL((attn_softmax_w<T, 8>), g, b, 0, s, P, Sm, Sd, nrows, S);
  else if (S <= 1024) hipLaunchKernelGGL((attn_softmax_w<T, 16>), g, b, 0, s, P, Sm, Sd, nrows, S);
  else if (S <= 2048) hipLaunchKernelGGL((attn_softmax_w<T, 32>), g, b, 0, s, P, Sm, Sd, nrows, S);
  else hipLaunchKernelGGL((attn_softmax_w<T, 64>), g, b, 0, s, P, Sm, Sd, nrows, S);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_attn_dsoftmax(PairT<T> dS, const T* Pm, const T* Pd, const float* dPm, const float* dPd, int nrows,
                                int S, hipStream_t s) {
  if (S > 4096) return hipErrorInvalidValue;
  const dim3 g(ceil_div(nrows, 4)), b(256);
  if (S <= 512) hipLaunchKernelGGL((attn_dsoftmax_w<T, 8>), g, b, 0, s, dS, Pm, Pd, dPm, dPd, nrows, S);
  else if (S <= 1024) hipLaunchKernelGGL((attn_dsoftmax_w<T, 16>), g, b, 0, s, dS, Pm, Pd, dPm, dPd, nrows, S);
  else if (S <= 2048) hipLaunchKernelGGL((attn_dsoftmax_w<T, 32>), g, b, 0, s, dS, Pm, Pd, dPm, dPd, nrows, S);
  else hipLaunchKernelGGL((attn_dsoftmax_w<T, 64>), g, b, 0, s, dS, Pm, Pd, dPm, dPd, nrows, S);
  return hipGetLastError();
}

hipError_t launch_group_sum(float* out, int64_t out_ld, const float* in, int T_, int Hk, int G, int dh, hipStream_t s) {
  hipLaunchKernelGGL(group_sum_kernel, dim3(grid_for((int64_t)T_ * Hk * dh)), dim3(NT), 0, s, out, out_ld, in, T_, Hk, G, dh);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_gelu_fwd(PairT<T> z, const T* um, const T* ud, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(gelu_fwd_kernel<T>, dim3(grid_for(n)), dim3(NT), 0, s, z, um, ud, n);
  return hipGetLastError();
}
template <typename T>
hipError_t launch_gelu_bwd(PairT<T> du, float* dudf, const T* um, const T* ud, const float* dzm, const float* dzd,
                           int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(gelu_bwd_kernel<T>, dim3(grid_for(n)), dim3(NT), 0, s, du, dudf, um, ud, dzm, dzd, n);
  return hipGetLastError();
}
template <typename T>
hipError_t launch_swiglu_fwd(PairT<T> z, const T* gum, const T* gud, int rows, int F, hipStream_t s) {
  if (F % 4 == 0 && rows <= 65535) {
    // workgroups of 128 threads divide the 1.3B row (1408 groups of 4) exactly
    const int nt = (F / 4) % 128 == 0 ? 128 : NT;
    hipLaunchKernelGGL(swiglu_fwd4_kernel<T>, dim3(ceil_div(F / 4, nt), rows), dim3(nt), 0, s, z, gum, gud, F);
  }
  else
    hipLaunchKernelGGL(swiglu_fwd_kernel<T>, dim3(grid_for((int64_t)rows * F)), dim3(NT), 0, s, z, gum, gud, rows, F);
  return hipGetLastError();
}
template <typename T>
hipError_t launch_swiglu_bwd(PairT<T> dgu, const T* gum, const T* gud, const float* dzm, const float* dzd, int rows,
                             int F, hipStream_t s) {
  if (F % 4 == 0 && rows <= 65535) {
    const int nt = (F / 4) % 128 == 0 ? 128 : NT;
    hipLaunchKernelGGL(swiglu_bwd4_kernel<T>, dim3(ceil_div(F / 4, nt), rows), dim3(nt), 0, s, dgu, gum, gud, dzm, dzd, F);
  }
  else
    hipLaunchKernelGGL(swiglu_bwd_kernel<T>, dim3(grid_for((int64_t)rows * F)), dim3(NT), 0, s, dgu, gum, gud, dzm, dzd, rows,
                       F);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_ce(PairT<T> dl, double* rowloss, const float* lm, const float* ld, const int32_t* tok,
                     const int32_t* lab, int T_, int S, int V, double inv_n, hipStream_t s) {
  hipLaunchKernelGGL(ce_kernel<T>, dim3(T_), dim3(NT), 0, s, dl, rowloss, lm, ld, tok, lab, T_, S, V, inv_n);
  return hipGetLastError();
}
hipError_t launch_loss_sum(double* out2, const double* rowloss, int T_, bool acc, hipStream_t s) {
  hipLaunchKernelGGL(loss_sum_kernel, dim3(1), dim3(NT), 0, s, out2, rowloss, T_, acc);
  return hipGetLastError();
}
hipError_t launch_count_targets(int64_t* out3, const int32_t* tok, const int32_t* lab, int B, int S, int V, hipStream_t s) {
  hipLaunchKernelGGL(count_targets_kernel, dim3(1), dim3(NT), 0, s, out3, tok, lab, B, S, V);
  return hipGetLastError();
}

hipError_t launch_token_sort(uint32_t* keys, const int32_t* tok, int T_, int V, hipStream_t s) {
  if (T_ > SORT_N) return hipErrorInvalidValue;
  hipLaunchKernelGGL(token_sort_kernel, dim3(1), dim3(1024), 0, s, keys, tok, T_, V);
  return hipGetLastError();
}
hipError_t launch_embed_bwd(float* hv, const uint32_t* keys, const float* dxd, int T_, int dm, double inv_eps, bool acc,
                            hipStream_t s) {
  hipLaunchKernelGGL(embed_bwd_kernel, dim3(T_, (dm + NT - 1) / NT), dim3(NT), 0, s, hv, keys, dxd, T_, dm, inv_eps,
                     acc);
  return hipGetLastError();
}
hipError_t launch_pos_bwd(float* hv, const float* dxd, int B, int S, int dm, double inv_eps, bool acc, hipStream_t s) {
  hipLaunchKernelGGL(pos_bwd_kernel, dim3(grid_for((int64_t)S * dm)), dim3(NT), 0, s, hv, dxd, B, S, dm, inv_eps, acc);
  return hipGetLastError();
}

#define INST_T(T)                                                                                                     \
  template hipError_t launch_cast_pair<T>(PairT<T>, const float*, const float*, int64_t, hipStream_t);                 \
  template hipError_t launch_embed_fwd<T>(PairF, const int32_t*, int, int, int, int, const T*, const float*, const T*, \
                                          const float*, double, int*, hipStream_t);                                    \
  template hipError_t launch_norm_fwd<T>(PairT<T>, const float*, const float*, int, int, bool, const T*, const float*, \
                                         const T*, const float*, double, float, hipStream_t);                          \
  template hipError_t launch_norm_bwd<T>(PairF, PairT<T>, const float*, const float*, const float*, const float*,      \
                                         const float*, const float*, int, int, bool, const T*, const float*, double,    \
                                         float, double*, double*, hipStream_t);                                        \
  template hipError_t launch_rope_inplace<T>(PairT<T>, int, int, int, int, int, const double*, hipStream_t);          \
  template hipError_t launch_qkv_bwd_post<T>(PairT<T>, float*, float*, int, int, int, int, int, const double*, bool,   \
                                             hipStream_t);                                                             \
  template hipError_t launch_attn_softmax<T>(PairT<T>, const float*, const float*, int, int, hipStream_t);             \
  template hipError_t launch_attn_dsoftmax<T>(PairT<T>, const T*, const T*, const float*, const float*, int, int,      \
                                              hipStream_t);                                                            \
  template hipError_t launch_gelu_fwd<T>(PairT<T>, const T*, const T*, int64_t, hipStream_t);                          \
  template hipError_t launch_gelu_bwd<T>(PairT<T>, float*, const T*, const T*, const float*, const float*,             \
                                         int64_t, hipStream_t);                                                        \
  template hipError_t launch_swiglu_fwd<T>(PairT<T>, const T*, const T*, int, int, hipStream_t);                       \
  template hipError_t launch_swiglu_bwd<T>(PairT<T>, const T*, const T*, const float*, const float*, int, int,         \
                                           hipStream_t);                                                               \
  template hipError_t launch_ce<T>(PairT<T>, double*, const float*, const float*, const int32_t*, const int32_t*, int, \
                                   int, int, double, hipStream_t);
INST_T(float)
INST_T(bf16_t)

}  // namespace fdh
