// Bandwidth-bound vector kernels over parameter-sized vectors: the perturbation
// operand, the quadratic test operator, the Lanczos recurrence with classical
// Gram-Schmidt (twice) reorthogonalisation against the stored Krylov basis,
// and per-layer block statistics.
//
// Reductions are deterministic: a fixed grid of RED_BLOCKS workgroups, each
// owning one contiguous chunk of the vector, accumulates fp32 products in
// fp64, reduces inside the workgroup in a fixed order and writes one partial
// per workgroup; a single-workgroup kernel then adds the partials in index
// order.  No floating-point atomics anywhere.
#include "kernels.h"

#include <type_traits>

namespace fdh {

namespace {

constexpr int NT = 256;

__host__ __device__ inline int64_t red_chunk(int64_t n) {
  int64_t c = (n + RED_BLOCKS - 1) / RED_BLOCKS;
  return (c + 1023) / 1024 * 1024;
}

unsigned grid_for(int64_t n) {
  int64_t g = (n + NT - 1) / NT;
  if (g > 65536) g = 65536;
  if (g < 1) g = 1;
  return (unsigned)g;
}

__global__ void fill_f32_kernel(float* p, int64_t n, float v) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) p[i] = v;
}
__global__ void fill_f64_kernel(double* p, int64_t n, double v) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) p[i] = v;
}

// lo = T(eps * v); with flag, flag[0] = 1 when some v[i] is NaN or infinite
template <typename T>
__global__ void scale_cast_kernel(T* lo, const float* v, double eps, int64_t n, int* flag) {
  bool bad = false;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    bad |= !isfinite(v[i]);
    stf(lo, i, (float)(eps * (double)v[i]));
  }
  if (flag && bad) flag[0] = 1;
}

template <typename T>
__global__ void quad_diag_kernel(const T* th, const float* d, const float* v, double eps, float* hv, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const double t = ldf(th, i), dd = d[i], vv = v[i];
    const double gp = dd * (t + eps * vv), gm = dd * (t - eps * vv);
    hv[i] = (float)((gp - gm) / (2.0 * eps));
  }
}

// ---- Lanczos ----------------------------------------------------------------
// Every pass works on groups of 8 consecutive elements per lane (two 16-byte
// loads of an fp32 vector, one of a bf16 basis row).  Workgroup chunks start at
// multiples of 1024 elements and basis rows at multiples of 8 (row stride
// ldq), so every full group is aligned; the group that crosses the end of the
// vector is loaded and stored element by element, with zeros past the end.
struct V8 { float x[8]; };
__device__ inline V8 ld8(const float* p, int64_t i) {
  const float4 a = *reinterpret_cast<const float4*>(p + i), b = *reinterpret_cast<const float4*>(p + i + 4);
  return V8{{a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w}};
}
__device__ inline V8 ld8(const bf16_t* p, int64_t i) {
  const uint4 u = *reinterpret_cast<const uint4*>(p + i);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
  V8 r;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    r.x[2 * t] = __uint_as_float(w[t] << 16);
    r.x[2 * t + 1] = __uint_as_float(w[t] & 0xFFFF0000u);
  }
  return r;
}
__device__ inline void st8(float* p, int64_t i, const V8& v) {
  *reinterpret_cast<float4*>(p + i) = make_float4(v.x[0], v.x[1], v.x[2], v.x[3]);
  *reinterpret_cast<float4*>(p + i + 4) = make_float4(v.x[4], v.x[5], v.x[6], v.x[7]);
}
__device__ inline void st8(bf16_t* p, int64_t i, const V8& v) {
  uint32_t w[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) w[t] = (uint32_t)f32_to_bf16(v.x[2 * t]) | ((uint32_t)f32_to_bf16(v.x[2 * t + 1]) << 16);
  *reinterpret_cast<uint4*>(p + i) = make_uint4(w[0], w[1], w[2], w[3]);
}
// ne < 8 valid elements (the tail group)
template <typename T> __device__ inline V8 ld8t(const T* p, int64_t i, int ne) {
  V8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r.x[e] = e < ne ? ldf(p, i + e) : 0.f;
  return r;
}
template <typename T> __device__ inline void st8t(T* p, int64_t i, const V8& v, int ne) {
#pragma unroll
  for (int e = 0; e < 8; ++e)
    if (e < ne) stf(p, i + e, v.x[e]);
}
// FULL: an aligned group of 8 (one branch-free vector access); otherwise the
// tail group, element by element.  Keeping the two apart keeps the main loops
// free of per-lane branches, so their loads issue back to back.
template <bool FULL, typename T> __device__ inline V8 ldv(const T* p, int64_t i, int ne) {
  if constexpr (FULL) return ld8(p, i);
  else return ld8t(p, i, ne);
}
template <bool FULL, typename T> __device__ inline void stv(T* p, int64_t i, const V8& v, int ne) {
  if constexpr (FULL) st8(p, i, v);
  else st8t(p, i, v, ne);
}
using Full = std::true_type;
using Tail = std::false_type;

// Runs body(i, 8, Full) over the full groups of [i0, s1) with stride `step`
// and body(i, s1 - i, Tail) for a final partial group of this lane.
template <typename F>
__device__ inline void for_groups(int64_t i0, int64_t s1, int64_t step, F&& body) {
  int64_t i = i0;
  for (; i + 8 <= s1; i += step) body(i, 8, Full{});
  if (i < s1) body(i, (int)(s1 - i), Tail{});
}

// Step A: w <- w - beta_{k-1} qprev ; partial = <w, q>
__global__ __launch_bounds__(NT) void lz_alpha_kernel(float* w, const float* q, const float* qprev, const double* beta,
                                                      int k, int64_t n, double* partial) {
  __shared__ double sh[NT / 64];
  const double bk = (k > 0) ? beta[k - 1] : 0.0;
  const int64_t ch = red_chunk(n);
  const int64_t s0 = blockIdx.x * ch, s1 = min(n, s0 + ch);
  double acc = 0.0;
  for_groups(s0 + 8 * threadIdx.x, s1, 8 * NT, [&](int64_t i, int ne, auto full) {
    constexpr bool F = decltype(full)::value;
    V8 wv = ldv<F>(w, i, ne);
    const V8 pv = ldv<F>(qprev, i, ne), qv = ldv<F>(q, i, ne);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      wv.x[e] = (float)((double)wv.x[e] - bk * (double)pv.x[e]);
      acc += (double)wv.x[e] * (double)qv.x[e];
    }
    stv<F>(w, i, wv, ne);
  });
  acc = block_sum<NT>(acc, sh);
  if (threadIdx.x == 0) partial[blockIdx.x] = acc;
}

// Step B (projections, with step A fused): w' = fp32(w - beta_{k-1} q_{k-1})
// is formed on the fly (not written; the update pass forms it again),
// alpha_k = <w', q_k>, p'_j = <w', Q_j> and g_j = <Q_new, Q_j> for the stored
// rows (Q_new = the row of q_k); the finish kernel takes p_j = p'_j - alpha_k g_j.
// One launch covers up to 32 rows: every wavefront of a workgroup takes all of
// them, [r0, r0 + nrl), over its own share of the chunk's 8-element groups
// (a lane keeps fp64 sums for 4 NG rows; rows are read in groups of 4 with
// their loads issued together), and the wavefronts' sums are added in a fixed
// order.  alpha's partial is formed by the launch with wa.
// partial[j * RED_BLOCKS + b] = p'_j, [(nv + j) * ...] = g_j, [2 nv * ...] = alpha part.
template <typename B, int NW, int NG>
__global__ __launch_bounds__(64 * NW, NG == 1 ? 4 : 1) void lz_project_kernel(const float* w, const float* q,
                                                             const float* qprev, const double* beta, int k,
                                                             BasisRows<B> R, int nv, int newest, int r0, int nrl,
                                                             bool wa, int64_t n, double* partial) {
  constexpr int RW = 4 * NG;
  __shared__ double red[NW][2 * RW + 1];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int nr = nrl;
  const int64_t ch = red_chunk(n);
  const int64_t s0 = blockIdx.x * ch, s1 = min(n, s0 + ch);
  const double bk = (k > 0) ? beta[k - 1] : 0.0;
  const B* rowp[RW];
#pragma unroll
  for (int r = 0; r < RW; ++r) rowp[r] = R.row(r0 + (r < nr ? r : 0));
  const B* qnp = R.row(newest);
  double pw[RW], pg[RW], pa = 0.0;
#pragma unroll
  for (int r = 0; r < RW; ++r) pw[r] = pg[r] = 0.0;
  for_groups(s0 + 512 * wave + 8 * lane, s1, 512 * NW, [&](int64_t i, int ne, auto full) {
    constexpr bool F = decltype(full)::value;
    const V8 wv = ldv<F>(w, i, ne), pv = ldv<F>(qprev, i, ne), qn = ldv<F>(qnp, i, ne);
    // w' = fp32(w - beta_{k-1} q_{k-1}), the alpha pass's rounding; alpha_k =
    // <w', q_k> (wavefront 0) and p_j = <w', Q_j> - alpha_k <Q_newest, Q_j>
    double w1[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) w1[e] = (double)(float)((double)wv.x[e] - bk * (double)pv.x[e]);
    if (wa) {
      const V8 qv = ldv<F>(q, i, ne);
#pragma unroll
      for (int e = 0; e < 8; ++e) pa = fma(w1[e], (double)qv.x[e], pa);
    }
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      if (4 * g < nr) {
        V8 rows[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) rows[t] = ldv<F>(rowp[4 * g + t], i, ne);
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const double x = rows[t].x[e];
            pw[4 * g + t] = fma(w1[e], x, pw[4 * g + t]);
            pg[4 * g + t] = fma((double)qn.x[e], x, pg[4 * g + t]);
          }
      }
    }
  });
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    if (r < nr) {
      const double tw = wave_sum(pw[r]), tg = wave_sum(pg[r]);
      if (lane == 0) {
        red[wave][r] = tw;
        red[wave][RW + r] = tg;
      }
    }
  }
  const double ta = wave_sum(pa);
  if (lane == 0) red[wave][2 * RW] = ta;
  __syncthreads();
  // partial columns: p'_j at j, g_j at nv + j, alpha's part at 2 nv
  const int t = threadIdx.x;
  if (t < 2 * nr + (wa ? 1 : 0)) {
    const int c = t < nr ? t : (t < 2 * nr ? RW + (t - nr) : 2 * RW);
    const int col = t < nr ? r0 + t : (t < 2 * nr ? nv + r0 + (t - nr) : 2 * nv);
    double sum = 0.0;
    for (int v = 0; v < NW; ++v) sum += red[v][c];
    partial[(int64_t)col * RED_BLOCKS + blockIdx.x] = sum;
  }
}

// Step C: w <- fp32(w1 - sum_j c_j Q_j) with w1 = fp32(w - alpha_k q) (nv >= 0
// rows, coefficients in coef), then partial = ||w||^2.  Rows are read in
// groups of 8 with their loads issued together; a group's rows past nv read
// row nv - 1 with coefficient zero.
template <typename B>
__global__ __launch_bounds__(NT) void lz_update_kernel(float* w, const float* q, const float* qprev, const double* beta,
                                                       int k, const double* alpha_k, BasisRows<B> R,
                                                       const double* coef, int nv, int64_t n, double* partial) {
  __shared__ double sh[NT / 64];
  __shared__ double cs[136];
  for (int j = threadIdx.x; j < 136; j += NT) cs[j] = j < nv ? coef[j] : 0.0;
  __syncthreads();
  const double a = *alpha_k;
  // with qprev the alpha pass was fused into the projection: w' = fp32(w -
  // beta_{k-1} q_{k-1}) is formed here again, with the same rounding
  const double bk = (qprev && k > 0) ? beta[k - 1] : 0.0;
  const int64_t ch = red_chunk(n);
  const int64_t s0 = blockIdx.x * ch, s1 = min(n, s0 + ch);
  double nrm = 0.0;
  for_groups(s0 + 8 * threadIdx.x, s1, 8 * NT, [&](int64_t i, int ne, auto full) {
    constexpr bool F = decltype(full)::value;
    V8 wv = ldv<F>(w, i, ne);
    const V8 qv = ldv<F>(q, i, ne);
    if (qprev) {
      const V8 pv = ldv<F>(qprev, i, ne);
#pragma unroll
      for (int e = 0; e < 8; ++e) wv.x[e] = (float)((double)wv.x[e] - bk * (double)pv.x[e]);
    }
    double acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = (double)(float)((double)wv.x[e] - a * (double)qv.x[e]);
    for (int j0 = 0; j0 < nv; j0 += 8) {
      V8 rows[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) rows[t] = ldv<F>(R.row(min(j0 + t, nv - 1)), i, ne);
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const double c = cs[j0 + t];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = fma(-c, (double)rows[t].x[e], acc[e]);
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      wv.x[e] = (float)acc[e];
      nrm += (double)wv.x[e] * (double)wv.x[e];
    }
    stv<F>(w, i, wv, ne);
  });
  nrm = block_sum<NT>(nrm, sh);
  if (threadIdx.x == 0) partial[blockIdx.x] = nrm;
}

// mode 0: alpha[k] = sum, update maxabs.
// mode 1: projections.  p_j and g_j (j < nv) are summed; row and column
//   `newest` of the Gram matrix G = Q^T Q of the stored rows are replaced by
//   g; then c = p + (p - G p) = 2 p - G p, the coefficients of both classical
//   Gram-Schmidt passes at once: the second pass's projections of
//   w - Q p are p - G p exactly (low-synchronisation CGS2, Swirydowicz et al.,
//   Numer. Linear Algebra Appl. 28, 2021).
// mode 2: beta[k] = sqrt(sum); breakdown test against tol * maxabs.
__global__ void lz_finish_kernel(LanczosDev st, int mode, int k, int nv, int newest, double tol) {
  __shared__ double sp[128];
  __shared__ double colsum[2 * 128 + 1];
  const int j = threadIdx.x;
  const int ncol = (mode == 1) ? 2 * nv + 1 : 1;
  // column sums of the partials in a fixed order: wavefront w takes columns
  // w, w + 4, ...; lane l adds partials l, l + 64, ..., then a fixed butterfly
  {
    const int wv = threadIdx.x >> 6, ln = threadIdx.x & 63;
    for (int c = wv; c < ncol; c += (int)(blockDim.x >> 6)) {
      double t = 0.0;
      for (int b = ln; b < RED_BLOCKS; b += 64) t += st.partial[(int64_t)c * RED_BLOCKS + b];
      t = wave_sum(t);
      if (ln == 0) colsum[c] = t;
    }
  }
  __syncthreads();
  double s = j < ncol ? colsum[j] : 0.0;
  if (mode == 1) {
    // alpha_k, and p_j = <w', Q_j> - alpha_k g_j with g_j = <Q_newest, Q_j>
    const double al = colsum[2 * nv];
    if (j == 0) {
      st.alpha[k] = al;
      st.maxabs[0] = fmax(st.maxabs[0], fabs(al));
    }
    if (j < nv) s -= al * colsum[nv + j];
  }
  if (mode == 0) {
    if (j == 0) {
      st.alpha[k] = s;
      st.maxabs[0] = fmax(st.maxabs[0], fabs(s));
    }
  } else if (mode == 1) {
    if (j < nv) sp[j] = s;
    if (j >= nv && j < 2 * nv) {
      st.gram[(int64_t)newest * 128 + (j - nv)] = s;
      st.gram[(int64_t)(j - nv) * 128 + newest] = s;
    }
    __syncthreads();
    if (j < nv) {
      double gp = 0.0;
      for (int i = 0; i < nv; ++i) gp += st.gram[(int64_t)j * 128 + i] * sp[i];
      st.coef[j] = 2.0 * sp[j] - gp;
    }
  } else if (j == 0) {
    const double b = sqrt(s);
    st.beta[k] = b;
    if (st.flag[0] == 0 && !(b > tol * st.maxabs[0])) st.flag[0] = k + 1;
  }
}

// Step D: beta_k from the last reduction; q_next = w / beta_k, the basis row
// (if any) = B(q_next) and the next HVP's perturbation operand (if any)
// lo = T(eps * q_next); after a breakdown all are zero.
template <typename B, typename T>
__global__ void lz_scale_kernel(const float* w, float* qn, B* row, T* lo, double eps, const double* beta_k, const int* flag,
                                int64_t n) {
  const bool broken = flag[0] != 0;
  const double inv = broken ? 0.0 : 1.0 / *beta_k;
  const int64_t step = 8 * (int64_t)gridDim.x * blockDim.x;
  for_groups(8 * (blockIdx.x * (int64_t)blockDim.x + threadIdx.x), n, step, [&](int64_t i, int ne, auto full) {
    constexpr bool F = decltype(full)::value;
    const V8 wv = ldv<F>(w, i, ne);
    V8 q, l;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      q.x[e] = (float)((double)wv.x[e] * inv);
      l.x[e] = (float)(eps * (double)q.x[e]);
    }
    stv<F>(qn, i, q, ne);
    if (row) stv<F>(row, i, q, ne);
    if (lo) stv<F>(lo, i, l, ne);
  });
}

// ---- conjugate gradient ------------------------------------------------------
// The vector steps of CG for (H + lam I) x = b (Hestenes-Stiefel), same
// chunked deterministic reductions as the Lanczos passes.  Scalars in sc:
// [0] (r, r), [1] (p, A p), [2] alpha, [3] (r_new, r_new), [4] beta.
// x = 0, r = p = b; partial = (b, b)
__global__ __launch_bounds__(NT) void cg_init_kernel(float* x, float* r, float* p, const float* b, int64_t n,
                                                     double* partial) {
  __shared__ double sh[NT / 64];
  const int64_t ch = red_chunk(n);
  const int64_t s0 = blockIdx.x * ch, s1 = min(n, s0 + ch);
  double acc = 0.0;
  for_groups(s0 + 8 * threadIdx.x, s1, 8 * NT, [&](int64_t i, int ne, auto full) {
    constexpr bool F = decltype(full)::value;
    const V8 bv = ldv<F>(b, i, ne);
    V8 z;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      z.x[e] = 0.f;
      acc += (double)bv.x[e] * (double)bv.x[e];
    }
    stv<F>(x, i, z, ne);
    stv<F>(r, i, bv, ne);
    stv<F>(p, i, bv, ne);
  });
  acc = block_sum<NT>(acc, sh);
  if (threadIdx.x == 0) partial[blockIdx.x] = acc;
}
// A p = H p + lam p (in place over H p); partial = (p, A p)
__global__ __launch_bounds__(NT) void cg_ap_kernel(float* ap, const float* p, double lam, int64_t n, double* partial) {
  __shared__ double sh[NT / 64];
  const int64_t ch = red_chunk(n);
  const int64_t s0 = blockIdx.x * ch, s1 = min(n, s0 + ch);
  double acc = 0.0;
  for_groups(s0 + 8 * threadIdx.x, s1, 8 * NT, [&](int64_t i, int ne, auto full) {
    constexpr bool F = decltype(full)::value;
    V8 av = ldv<F>(ap, i, ne);
    const V8 pv = ldv<F>(p, i, ne);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      av.x[e] = (float)((double)av.x[e] + lam * (double)pv.x[e]);
      acc += (double)pv.x[e] * (double)av.x[e];
    }
    stv<F>(ap, i, av, ne);
  });
  acc = block_sum<NT>(acc, sh);
  if (threadIdx.x == 0) partial[blockIdx.x] = acc;
}
// x += alpha p, r -= alpha A p; partial = (r, r)
__global__ __launch_bounds__(NT) void cg_step_kernel(float* x, float* r, const float* p, const float* ap,
                                                     const double* sc, int64_t n, double* partial) {
  __shared__ double sh[NT / 64];
  const double alpha = sc[2];
  const int64_t ch = red_chunk(n);
  const int64_t s0 = blockIdx.x * ch, s1 = min(n, s0 + ch);
  double acc = 0.0;
  for_groups(s0 + 8 * threadIdx.x, s1, 8 * NT, [&](int64_t i, int ne, auto full) {
    constexpr bool F = decltype(full)::value;
    V8 xv = ldv<F>(x, i, ne), rv = ldv<F>(r, i, ne);
    const V8 pv = ldv<F>(p, i, ne), av = ldv<F>(ap, i, ne);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      xv.x[e] = (float)((double)xv.x[e] + alpha * (double)pv.x[e]);
      rv.x[e] = (float)((double)rv.x[e] - alpha * (double)av.x[e]);
      acc += (double)rv.x[e] * (double)rv.x[e];
    }
    stv<F>(x, i, xv, ne);
    stv<F>(r, i, rv, ne);
  });
  acc = block_sum<NT>(acc, sh);
  if (threadIdx.x == 0) partial[blockIdx.x] = acc;
}
// p = r + beta p, and the next HVP's perturbation operand lo = T(eps p) if lo
template <typename T>
__global__ void cg_dir_kernel(float* p, const float* r, const double* sc, T* lo, double eps, int64_t n) {
  const double beta = sc[4];
  const int64_t step = 8 * (int64_t)gridDim.x * blockDim.x;
  for_groups(8 * (blockIdx.x * (int64_t)blockDim.x + threadIdx.x), n, step, [&](int64_t i, int ne, auto full) {
    constexpr bool F = decltype(full)::value;
    V8 pv = ldv<F>(p, i, ne);
    const V8 rv = ldv<F>(r, i, ne);
    V8 l;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      pv.x[e] = (float)((double)rv.x[e] + beta * (double)pv.x[e]);
      l.x[e] = (float)(eps * (double)pv.x[e]);
    }
    stv<F>(p, i, pv, ne);
    if (lo) stv<F>(lo, i, l, ne);
  });
}
// mode 0: sc[0] = sum.  mode 1: sc[1] = sum, sc[2] = sc[0] / sum (0 unless sum > 0).
// mode 2: sc[3] = sum, sc[4] = sum / sc[0] (0 if sc[0] == 0), sc[0] = sum.
__global__ void cg_finish_kernel(double* sc, const double* partial, int mode) {
  // one wavefront: lane l adds partials l, l + 64, ... in order, then a fixed butterfly
  double t = 0.0;
  for (int b = threadIdx.x; b < RED_BLOCKS; b += 64) t += partial[b];
  const double s = wave_sum(t);
  if (threadIdx.x != 0) return;
  if (mode == 0) {
    sc[0] = s;
  } else if (mode == 1) {
    sc[1] = s;
    sc[2] = s > 0.0 ? sc[0] / s : 0.0;
  } else {
    sc[3] = s;
    sc[4] = sc[0] > 0.0 ? s / sc[0] : 0.0;
    sc[0] = s;
  }
}

// lo = T(eps * v), 8 elements per lane (16-byte aligned operands); with flag,
// flag[0] = 1 when some v[i] is NaN or infinite (elements past the end load as 0)
template <typename T>
__global__ void scale_cast8_kernel(T* lo, const float* v, double eps, int64_t n, int* flag) {
  const int64_t step = 8 * (int64_t)gridDim.x * blockDim.x;
  bool bad = false;
  for_groups(8 * (blockIdx.x * (int64_t)blockDim.x + threadIdx.x), n, step, [&](int64_t i, int ne, auto full) {
    constexpr bool F = decltype(full)::value;
    V8 x = ldv<F>(v, i, ne);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      bad |= !isfinite(x.x[e]);
      x.x[e] = (float)(eps * (double)x.x[e]);
    }
    stv<F>(lo, i, x, ne);
  });
  if (flag && bad) flag[0] = 1;
}

// flag[0] = 1 when some x[i] is NaN or infinite (one read of x)
__global__ void nonfinite_scan8_kernel(const float* x, int64_t n, int* flag) {
  const int64_t step = 8 * (int64_t)gridDim.x * blockDim.x;
  bool bad = false;
  for_groups(8 * (blockIdx.x * (int64_t)blockDim.x + threadIdx.x), n, step, [&](int64_t i, int ne, auto full) {
    constexpr bool F = decltype(full)::value;
    const V8 v = ldv<F>(x, i, ne);
#pragma unroll
    for (int e = 0; e < 8; ++e) bad |= !isfinite(v.x[e]);
  });
  if (bad) flag[0] = 1;
}
__global__ void nonfinite_scan_kernel(const float* x, int64_t n, int* flag) {
  bool bad = false;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    bad |= !isfinite(x[i]);
  if (bad) flag[0] = 1;
}

// sums over [s0, s1): ||a||^2, ||b||^2, <a, b>, ||a - b||^2
__global__ void range_dots_kernel(const float* a, const float* b, int64_t s0, int64_t s1, double* partial) {
  __shared__ double sh[NT / 64];
  double aa = 0.0, bb = 0.0, ab = 0.0, dd = 0.0;
  for (int64_t i = s0 + blockIdx.x * (int64_t)NT + threadIdx.x; i < s1; i += (int64_t)gridDim.x * NT) {
    const double x = a[i], y = b[i];
    aa += x * x;
    bb += y * y;
    ab += x * y;
    dd += (x - y) * (x - y);
  }
  aa = block_sum<NT>(aa, sh);
  bb = block_sum<NT>(bb, sh);
  ab = block_sum<NT>(ab, sh);
  dd = block_sum<NT>(dd, sh);
  if (threadIdx.x == 0) {
    partial[blockIdx.x * 4 + 0] = aa;
    partial[blockIdx.x * 4 + 1] = bb;
    partial[blockIdx.x * 4 + 2] = ab;
    partial[blockIdx.x * 4 + 3] = dd;
  }
}

__global__ void range_dots_finish(const double* partial, int nb, double* out) {
  const int c = threadIdx.x;
  if (c >= 4) return;
  double s = 0.0;
  for (int b = 0; b < nb; ++b) s += partial[b * 4 + c];
  out[c] = s;
}

__global__ void mask_range_kernel(float* out, const float* v, int64_t s0, int64_t s1, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    out[i] = (i >= s0 && i < s1) ? v[i] : 0.f;
}

}  // namespace

hipError_t launch_fill_f32(float* p, int64_t n, float v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_f32_kernel, dim3(grid_for(n)), dim3(NT), 0, s, p, n, v);
  return hipGetLastError();
}
namespace {
__global__ void copy16_kernel(uint4* dst, const uint4* src, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}
}  // namespace

hipError_t launch_copy16(void* dst, const void* src, size_t bytes, hipStream_t s) {
  const int64_t n = (int64_t)(bytes / 16);
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(copy16_kernel, dim3(grid_for(n)), dim3(NT), 0, s, (uint4*)dst, (const uint4*)src, n);
  return hipGetLastError();
}

namespace {
// out = sum of the ns partial products in slice order (acc: out += that sum)
__global__ void sum_splits_kernel(float* out, const float* part, int ns, int64_t n, bool acc) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    double t = 0.0;
    for (int j = 0; j < ns; ++j) t += (double)part[(int64_t)j * n + i];
    out[i] = acc ? out[i] + (float)t : (float)t;
  }
}
__global__ void sum_splits4_kernel(float4* out, const float4* part, int ns, int64_t n4, bool acc) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n4; i += (int64_t)gridDim.x * blockDim.x) {
    double t[4] = {0.0, 0.0, 0.0, 0.0};
    for (int j = 0; j < ns; ++j) {
      const float4 p = part[(int64_t)j * n4 + i];
      t[0] += p.x; t[1] += p.y; t[2] += p.z; t[3] += p.w;
    }
    float4 r = make_float4((float)t[0], (float)t[1], (float)t[2], (float)t[3]);
    if (acc) {
      const float4 o = out[i];
      r.x += o.x; r.y += o.y; r.z += o.z; r.w += o.w;
    }
    out[i] = r;
  }
}
}  // namespace

hipError_t launch_sum_splits(float* out, const float* part, int ns, int64_t n, bool acc, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (n % 4 == 0 && (uintptr_t)out % 16 == 0 && (uintptr_t)part % 16 == 0)
    hipLaunchKernelGGL(sum_splits4_kernel, dim3(grid_for(n / 4)), dim3(NT), 0, s, (float4*)out, (const float4*)part, ns,
                       n / 4, acc);
  else
    hipLaunchKernelGGL(sum_splits_kernel, dim3(grid_for(n)), dim3(NT), 0, s, out, part, ns, n, acc);
  return hipGetLastError();
}

hipError_t launch_fill_f64(double* p, int64_t n, double v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_f64_kernel, dim3(grid_for(n)), dim3(NT), 0, s, p, n, v);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_scale_cast(T* lo, const float* v, double eps, int64_t n, hipStream_t s, int* nonfinite) {
  if (n <= 0) return hipSuccess;
  if ((uintptr_t)lo % 16 == 0 && (uintptr_t)v % 16 == 0)
    hipLaunchKernelGGL(scale_cast8_kernel<T>, dim3(grid_for((n + 7) / 8)), dim3(NT), 0, s, lo, v, eps, n, nonfinite);
  else
    hipLaunchKernelGGL(scale_cast_kernel<T>, dim3(grid_for(n)), dim3(NT), 0, s, lo, v, eps, n, nonfinite);
  return hipGetLastError();
}
template hipError_t launch_scale_cast<float>(float*, const float*, double, int64_t, hipStream_t, int*);
template hipError_t launch_scale_cast<bf16_t>(bf16_t*, const float*, double, int64_t, hipStream_t, int*);

hipError_t launch_nonfinite_scan(const float* x, int64_t n, int* flag, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if ((uintptr_t)x % 16 == 0)
    hipLaunchKernelGGL(nonfinite_scan8_kernel, dim3(grid_for((n + 7) / 8)), dim3(NT), 0, s, x, n, flag);
  else
    hipLaunchKernelGGL(nonfinite_scan_kernel, dim3(grid_for(n)), dim3(NT), 0, s, x, n, flag);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_quad_diag_hvp(const T* theta, const float* d, const float* v, double eps, float* hv, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(quad_diag_kernel<T>, dim3(grid_for(n)), dim3(NT), 0, s, theta, d, v, eps, hv, n);
  return hipGetLastError();
}
template hipError_t launch_quad_diag_hvp<float>(const float*, const float*, const float*, double, float*, int64_t, hipStream_t);
template hipError_t launch_quad_diag_hvp<bf16_t>(const bf16_t*, const float*, const float*, double, float*, int64_t, hipStream_t);

hipError_t launch_lanczos_alpha(float* w, const float* q, const float* qprev, LanczosDev st, int k, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(lz_alpha_kernel, dim3(RED_BLOCKS), dim3(NT), 0, s, w, q, qprev, st.beta, k, n, st.partial);
  hipLaunchKernelGGL(lz_finish_kernel, dim3(1), dim3(256), 0, s, st, 0, k, 1, 0, 0.0);
  return hipGetLastError();
}

template <typename B>
hipError_t launch_lanczos_project(const float* w, const float* q, const float* qprev, BasisRows<B> rows, int nv, int newest,
                                  LanczosDev st, int k, int64_t n, hipStream_t s) {
  if (nv < 1 || nv > 128 || newest < 0 || newest >= nv) return hipErrorInvalidValue;
#define LZP(W, G, R0, NRL, WA)                                                                                     \
  hipLaunchKernelGGL((lz_project_kernel<B, W, G>), dim3(RED_BLOCKS), dim3(64 * W), 0, s, w, q, qprev,                 \
                     (const double*)st.beta, k, rows, nv, newest, R0, NRL, WA, n, st.partial)
  // element split over up to 32 rows per launch (further launches for the
  // next 32 rows each, without alpha)
  auto es = [&](int r0, int nrl, bool wa) {
    if (nrl <= 4) LZP(4, 1, r0, nrl, wa);
    else if (nrl <= 8) LZP(4, 2, r0, nrl, wa);
    else if (nrl <= 16) LZP(4, 4, r0, nrl, wa);
    else if (nrl <= 24) LZP(4, 6, r0, nrl, wa);
    else LZP(4, 8, r0, nrl, wa);
  };
  for (int r0 = 0; r0 < nv; r0 += 32) es(r0, std::min(32, nv - r0), r0 == 0);
#undef LZP
  hipLaunchKernelGGL(lz_finish_kernel, dim3(1), dim3(256), 0, s, st, 1, k, nv, newest, 0.0);
  return hipGetLastError();
}

template <typename B>
hipError_t launch_lanczos_update(float* w, const float* q, const float* qprev, BasisRows<B> rows, int nv, LanczosDev st,
                                 int k, int64_t n, hipStream_t s) {
  if (nv < 0 || nv > 128) return hipErrorInvalidValue;
  hipLaunchKernelGGL(lz_update_kernel<B>, dim3(RED_BLOCKS), dim3(NT), 0, s, w, q, qprev, (const double*)st.beta, k,
                     (const double*)(st.alpha + k), rows, (const double*)st.coef, nv, n, st.partial);
  return hipGetLastError();
}

template <typename B, typename T>
hipError_t launch_lanczos_normalise(const float* w, float* qnext, B* basis_row, T* lo, double eps, LanczosDev st, int k, double tol,
                                    int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(lz_finish_kernel, dim3(1), dim3(256), 0, s, st, 2, k, 1, 0, tol);
  hipLaunchKernelGGL((lz_scale_kernel<B, T>), dim3(grid_for((n + 7) / 8)), dim3(NT), 0, s, w, qnext, basis_row, lo, eps,
                     (const double*)(st.beta + k), (const int*)st.flag, n);
  return hipGetLastError();
}

#define INST_LZ(B)                                                                                                   \
  template hipError_t launch_lanczos_project<B>(const float*, const float*, const float*, BasisRows<B>, int, int,      \
                                                LanczosDev, int, int64_t, hipStream_t);                               \
  template hipError_t launch_lanczos_update<B>(float*, const float*, const float*, BasisRows<B>, int, LanczosDev, int, \
                                               int64_t, hipStream_t);                                                 \
  template hipError_t launch_lanczos_normalise<B, float>(const float*, float*, B*, float*, double, LanczosDev, int, double,   \
                                                         int64_t, hipStream_t);                                              \
  template hipError_t launch_lanczos_normalise<B, bf16_t>(const float*, float*, B*, bf16_t*, double, LanczosDev, int, double, \
                                                          int64_t, hipStream_t);
INST_LZ(float)
INST_LZ(bf16_t)

hipError_t launch_cg_init(float* x, float* r, float* p, const float* b, double* sc, double* partial, int64_t n,
                          hipStream_t s) {
  hipLaunchKernelGGL(cg_init_kernel, dim3(RED_BLOCKS), dim3(NT), 0, s, x, r, p, b, n, partial);
  hipLaunchKernelGGL(cg_finish_kernel, dim3(1), dim3(64), 0, s, sc, (const double*)partial, 0);
  return hipGetLastError();
}
hipError_t launch_cg_ap(float* ap, const float* p, double lam, double* sc, double* partial, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(cg_ap_kernel, dim3(RED_BLOCKS), dim3(NT), 0, s, ap, p, lam, n, partial);
  hipLaunchKernelGGL(cg_finish_kernel, dim3(1), dim3(64), 0, s, sc, (const double*)partial, 1);
  return hipGetLastError();
}
hipError_t launch_cg_step(float* x, float* r, const float* p, const float* ap, double* sc, double* partial, int64_t n,
                          hipStream_t s) {
  hipLaunchKernelGGL(cg_step_kernel, dim3(RED_BLOCKS), dim3(NT), 0, s, x, r, p, ap, (const double*)sc, n, partial);
  hipLaunchKernelGGL(cg_finish_kernel, dim3(1), dim3(64), 0, s, sc, (const double*)partial, 2);
  return hipGetLastError();
}
template <typename T>
hipError_t launch_cg_dir(float* p, const float* r, const double* sc, T* lo, double eps, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(cg_dir_kernel<T>, dim3(grid_for((n + 7) / 8)), dim3(NT), 0, s, p, r, sc, lo, eps, n);
  return hipGetLastError();
}
template hipError_t launch_cg_dir<float>(float*, const float*, const double*, float*, double, int64_t, hipStream_t);
template hipError_t launch_cg_dir<bf16_t>(float*, const float*, const double*, bf16_t*, double, int64_t, hipStream_t);

hipError_t launch_block_stats(const float* a, const float* b, const int64_t* ranges, int nblk, double* partial, double* out, hipStream_t s) {
  // ranges: host array [nblk][2]; partial: device [256 * 4]; out: device [nblk * 4]
  for (int i = 0; i < nblk; ++i) {
    hipLaunchKernelGGL(range_dots_kernel, dim3(256), dim3(NT), 0, s, a, b, ranges[2 * i], ranges[2 * i + 1], partial);
    hipLaunchKernelGGL(range_dots_finish, dim3(1), dim3(64), 0, s, (const double*)partial, 256, out + 4 * i);
  }
  return hipGetLastError();
}

hipError_t launch_mask_range(float* out, const float* v, int64_t s0, int64_t s1, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(mask_range_kernel, dim3(grid_for(n)), dim3(NT), 0, s, out, v, s0, s1, n);
  return hipGetLastError();
}

}  // namespace fdh
