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

namespace fdh {

namespace {

constexpr int NT = 256;
constexpr int JG = 16;   // basis rows reduced per sweep (fp64 accumulators per thread)

__host__ __device__ inline int64_t red_chunk(int64_t n) {
  int64_t c = (n + RED_BLOCKS - 1) / RED_BLOCKS;
  return (c + 1023) / 1024 * 1024;
}

template <typename B> __device__ inline float ldb(const B* p, int64_t i) { return ldf(p, i); }

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

template <typename T>
__global__ void scale_cast_kernel(T* lo, const float* v, double eps, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    stf(lo, i, (float)(eps * (double)v[i]));
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
// Step A: w <- w - beta_k qprev ; partial = <w, q>
__global__ void lz_alpha_kernel(float* w, const float* q, const float* qprev, const double* beta, int k,
                                int64_t n, double* partial) {
  __shared__ double sh[NT / 64];
  const double bk = (k > 0) ? beta[k - 1] : 0.0;
  const int64_t ch = red_chunk(n);
  const int64_t s0 = blockIdx.x * ch, s1 = min(n, s0 + ch);
  double acc = 0.0;
  for (int64_t i = s0 + threadIdx.x; i < s1; i += NT) {
    const float wi = (float)((double)w[i] - bk * (double)qprev[i]);
    w[i] = wi;
    acc += (double)wi * (double)q[i];
  }
  acc = block_sum<NT>(acc, sh);
  if (threadIdx.x == 0) partial[blockIdx.x] = acc;
}

// 4-element groups: float4 for fp32 vectors, 4 basis entries (8 or 16 bytes)
struct F4 { float x[4]; };
__device__ inline F4 ld4(const float* p, int64_t i) {
  const float4 v = *reinterpret_cast<const float4*>(p + i);
  return F4{{v.x, v.y, v.z, v.w}};
}
__device__ inline void st4(float* p, int64_t i, const F4& f) {
  *reinterpret_cast<float4*>(p + i) = make_float4(f.x[0], f.x[1], f.x[2], f.x[3]);
}
__device__ inline F4 ld4(const bf16_t* p, int64_t i) {
  const uint2 u = *reinterpret_cast<const uint2*>(p + i);
  return F4{{bf16_to_f32((bf16_t)(u.x & 0xFFFF)), bf16_to_f32((bf16_t)(u.x >> 16)), bf16_to_f32((bf16_t)(u.y & 0xFFFF)),
             bf16_to_f32((bf16_t)(u.y >> 16))}};
}
__device__ inline void st4(bf16_t* p, int64_t i, const F4& f) {
  uint2 u;
  u.x = (uint32_t)f32_to_bf16(f.x[0]) | ((uint32_t)f32_to_bf16(f.x[1]) << 16);
  u.y = (uint32_t)f32_to_bf16(f.x[2]) | ((uint32_t)f32_to_bf16(f.x[3]) << 16);
  *reinterpret_cast<uint2*>(p + i) = u;
}

// Vectorised pass (n % 4 == 0): each thread owns groups of 4 consecutive
// elements of its workgroup's chunk.  Same arithmetic as lz_pass_kernel.
template <typename B>
__global__ __launch_bounds__(NT) void lz_pass4_kernel(float* w, const float* x, const double* a_src, const double* c_src,
                                                      int nv_upd, const B* basis, int nv_proj, int64_t n,
                                                      double* partial) {
  __shared__ double sh[NT / 64];
  __shared__ double cs[128];
  const int64_t ch = red_chunk(n);
  const int64_t s0 = blockIdx.x * ch, s1 = min(n, s0 + ch);
  const double a = a_src ? *a_src : 0.0;
  for (int j = threadIdx.x; j < nv_upd; j += NT) cs[j] = c_src[j];
  __syncthreads();
  if (x || nv_upd > 0) {
    for (int64_t i = s0 + 4 * threadIdx.x; i < s1; i += 4 * NT) {
      F4 wv = ld4(w, i);
      double acc4[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) acc4[e] = wv.x[e];
      if (x) {
        const F4 xv = ld4(x, i);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc4[e] -= a * (double)xv.x[e];
      }
      for (int j = 0; j < nv_upd; ++j) {
        const F4 q = ld4(basis, (int64_t)j * n + i);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc4[e] -= cs[j] * (double)q.x[e];
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) wv.x[e] = (float)acc4[e];
      st4(w, i, wv);
    }
  }
  if (nv_proj == 0) {
    double acc = 0.0;
    for (int64_t i = s0 + 4 * threadIdx.x; i < s1; i += 4 * NT) {
      const F4 wv = ld4(w, i);
#pragma unroll
      for (int e = 0; e < 4; ++e) acc += (double)wv.x[e] * (double)wv.x[e];
    }
    acc = block_sum<NT>(acc, sh);
    if (threadIdx.x == 0) partial[blockIdx.x] = acc;
    return;
  }
  for (int j0 = 0; j0 < nv_proj; j0 += JG) {
    double acc[JG];
#pragma unroll
    for (int j = 0; j < JG; ++j) acc[j] = 0.0;
    const int nj = min(JG, nv_proj - j0);
    for (int64_t i = s0 + 4 * threadIdx.x; i < s1; i += 4 * NT) {
      const F4 wv = ld4(w, i);
#pragma unroll
      for (int j = 0; j < JG; ++j)
        if (j < nj) {
          const F4 q = ld4(basis, (int64_t)(j0 + j) * n + i);
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[j] += (double)wv.x[e] * (double)q.x[e];
        }
    }
    for (int j = 0; j < nj; ++j) {
      const double t = block_sum<NT>(acc[j], sh);
      if (threadIdx.x == 0) partial[(int64_t)(j0 + j) * RED_BLOCKS + blockIdx.x] = t;
    }
  }
}

__global__ __launch_bounds__(NT) void lz_alpha4_kernel(float* w, const float* q, const float* qprev, const double* beta,
                                                       int k, int64_t n, double* partial) {
  __shared__ double sh[NT / 64];
  const double bk = (k > 0) ? beta[k - 1] : 0.0;
  const int64_t ch = red_chunk(n);
  const int64_t s0 = blockIdx.x * ch, s1 = min(n, s0 + ch);
  double acc = 0.0;
  for (int64_t i = s0 + 4 * threadIdx.x; i < s1; i += 4 * NT) {
    F4 wv = ld4(w, i);
    const F4 pv = ld4(qprev, i), qv = ld4(q, i);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      wv.x[e] = (float)((double)wv.x[e] - bk * (double)pv.x[e]);
      acc += (double)wv.x[e] * (double)qv.x[e];
    }
    st4(w, i, wv);
  }
  acc = block_sum<NT>(acc, sh);
  if (threadIdx.x == 0) partial[blockIdx.x] = acc;
}

template <typename B>
__global__ void lz_scale4_kernel(const float* w, float* qn, B* row, const double* beta_k, const int* flag, int64_t n) {
  const bool broken = flag[0] != 0;
  const double inv = broken ? 0.0 : 1.0 / *beta_k;
  const int64_t n4 = n / 4;
  for (int64_t g = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; g < n4; g += (int64_t)gridDim.x * blockDim.x) {
    const F4 wv = ld4(w, 4 * g);
    F4 q;
#pragma unroll
    for (int e = 0; e < 4; ++e) q.x[e] = (float)((double)wv.x[e] * inv);
    st4(qn, 4 * g, q);
    if (row) st4(row, 4 * g, q);
  }
}

// Generic pass: w <- w - a*x - sum_j c_j Q_j (any part optional), then either
// partial[j] = <w, Q_j> for j < nv_proj, or partial[0] = ||w||^2 when nv_proj == 0.
template <typename B>
__global__ void lz_pass_kernel(float* w, const float* x, const double* a_src, const double* c_src, int nv_upd,
                               const B* basis, int nv_proj, int64_t n, double* partial) {
  __shared__ double sh[NT / 64];
  __shared__ double cs[128];
  const int64_t ch = red_chunk(n);
  const int64_t s0 = blockIdx.x * ch, s1 = min(n, s0 + ch);
  const double a = a_src ? *a_src : 0.0;
  for (int j = threadIdx.x; j < nv_upd; j += NT) cs[j] = c_src[j];
  __syncthreads();
  if (x || nv_upd > 0) {
    for (int64_t i = s0 + threadIdx.x; i < s1; i += NT) {
      double wi = w[i];
      if (x) wi -= a * (double)x[i];
      for (int j = 0; j < nv_upd; ++j) wi -= cs[j] * (double)ldb(basis, (int64_t)j * n + i);
      w[i] = (float)wi;
    }
  }
  if (nv_proj == 0) {
    double acc = 0.0;
    for (int64_t i = s0 + threadIdx.x; i < s1; i += NT) {
      const double wi = w[i];
      acc += wi * wi;
    }
    acc = block_sum<NT>(acc, sh);
    if (threadIdx.x == 0) partial[blockIdx.x] = acc;
    return;
  }
  for (int j0 = 0; j0 < nv_proj; j0 += JG) {
    double acc[JG];
#pragma unroll
    for (int j = 0; j < JG; ++j) acc[j] = 0.0;
    const int nj = min(JG, nv_proj - j0);
    for (int64_t i = s0 + threadIdx.x; i < s1; i += NT) {
      const double wi = w[i];
#pragma unroll
      for (int j = 0; j < JG; ++j)
        if (j < nj) acc[j] += wi * (double)ldb(basis, (int64_t)(j0 + j) * n + i);
    }
    for (int j = 0; j < nj; ++j) {
      const double t = block_sum<NT>(acc[j], sh);
      if (threadIdx.x == 0) partial[(int64_t)(j0 + j) * RED_BLOCKS + blockIdx.x] = t;
    }
  }
}

// mode 0: alpha[k] = sum, update maxabs.  mode 1: coef[dst + j] = sum_j for j < nv.
// mode 2: beta[k] = sqrt(sum); breakdown test against tol * maxabs.
__global__ void lz_finish_kernel(LanczosDev st, int mode, int k, int nv, int dst, double tol) {
  const int j = threadIdx.x;
  const int ncol = (mode == 1) ? nv : 1;
  if (j >= ncol) return;
  double s = 0.0;
  for (int b = 0; b < RED_BLOCKS; ++b) s += st.partial[(int64_t)j * RED_BLOCKS + b];
  if (mode == 0) {
    st.alpha[k] = s;
    st.maxabs[0] = fmax(st.maxabs[0], fabs(s));
  } else if (mode == 1) {
    st.coef[dst + j] = s;
  } else {
    const double b = sqrt(s);
    st.beta[k] = b;
    if (st.flag[0] == 0 && !(b > tol * st.maxabs[0])) st.flag[0] = k + 1;
  }
}

template <typename B>
__global__ void lz_scale_kernel(const float* w, float* qn, B* row, const double* beta_k, const int* flag, int64_t n) {
  const bool broken = flag[0] != 0;
  const double inv = broken ? 0.0 : 1.0 / *beta_k;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const float q = (float)((double)w[i] * inv);
    qn[i] = q;
    if (row) stf(row, i, q);
  }
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

hipError_t launch_fill_f64(double* p, int64_t n, double v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_f64_kernel, dim3(grid_for(n)), dim3(NT), 0, s, p, n, v);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_scale_cast(T* lo, const float* v, double eps, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(scale_cast_kernel<T>, dim3(grid_for(n)), dim3(NT), 0, s, lo, v, eps, n);
  return hipGetLastError();
}
template hipError_t launch_scale_cast<float>(float*, const float*, double, int64_t, hipStream_t);
template hipError_t launch_scale_cast<bf16_t>(bf16_t*, const float*, double, int64_t, hipStream_t);

template <typename T>
hipError_t launch_quad_diag_hvp(const T* theta, const float* d, const float* v, double eps, float* hv, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(quad_diag_kernel<T>, dim3(grid_for(n)), dim3(NT), 0, s, theta, d, v, eps, hv, n);
  return hipGetLastError();
}
template hipError_t launch_quad_diag_hvp<float>(const float*, const float*, const float*, double, float*, int64_t, hipStream_t);
template hipError_t launch_quad_diag_hvp<bf16_t>(const bf16_t*, const float*, const float*, double, float*, int64_t, hipStream_t);

hipError_t launch_lanczos_alpha(float* w, const float* q, const float* qprev, LanczosDev st, int k, int64_t n, hipStream_t s) {
  if (n % 4 == 0)
    hipLaunchKernelGGL(lz_alpha4_kernel, dim3(RED_BLOCKS), dim3(NT), 0, s, w, q, qprev, st.beta, k, n, st.partial);
  else
    hipLaunchKernelGGL(lz_alpha_kernel, dim3(RED_BLOCKS), dim3(NT), 0, s, w, q, qprev, st.beta, k, n, st.partial);
  hipLaunchKernelGGL(lz_finish_kernel, dim3(1), dim3(256), 0, s, st, 0, k, 1, 0, 0.0);
  return hipGetLastError();
}

template <typename B>
hipError_t launch_lanczos_b(float* w, const float* q, const B* basis, int nv, LanczosDev st, int k, int64_t n, hipStream_t s) {
  if (n % 4 == 0)
    hipLaunchKernelGGL(lz_pass4_kernel<B>, dim3(RED_BLOCKS), dim3(NT), 0, s, w, q, (const double*)(st.alpha + k),
                       (const double*)nullptr, 0, basis, nv, n, st.partial);
  else
    hipLaunchKernelGGL(lz_pass_kernel<B>, dim3(RED_BLOCKS), dim3(NT), 0, s, w, q, (const double*)(st.alpha + k),
                       (const double*)nullptr, 0, basis, nv, n, st.partial);
  if (nv > 0) hipLaunchKernelGGL(lz_finish_kernel, dim3(1), dim3(256), 0, s, st, 1, k, nv, 0, 0.0);
  return hipGetLastError();
}

template <typename B>
hipError_t launch_lanczos_cgs(float* w, const B* basis, int nv, LanczosDev st, int pass, bool last, int k, int64_t n, hipStream_t s) {
  // coefficients of this pass live at coef[pass * 128]; the next pass writes coef[(pass+1) * 128]
  if (n % 4 == 0)
    hipLaunchKernelGGL(lz_pass4_kernel<B>, dim3(RED_BLOCKS), dim3(NT), 0, s, w, (const float*)nullptr, (const double*)nullptr,
                       (const double*)(st.coef + pass * 128), nv, basis, last ? 0 : nv, n, st.partial);
  else
  hipLaunchKernelGGL(lz_pass_kernel<B>, dim3(RED_BLOCKS), dim3(NT), 0, s, w, (const float*)nullptr, (const double*)nullptr,
                     (const double*)(st.coef + pass * 128), nv, basis, last ? 0 : nv, n, st.partial);
  if (!last) hipLaunchKernelGGL(lz_finish_kernel, dim3(1), dim3(256), 0, s, st, 1, k, nv, (pass + 1) * 128, 0.0);
  return hipGetLastError();
}

template <typename B>
hipError_t launch_lanczos_normalise(const float* w, float* qnext, B* basis_row, LanczosDev st, int k, double tol, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(lz_finish_kernel, dim3(1), dim3(256), 0, s, st, 2, k, 1, 0, tol);
  if (n % 4 == 0)
    hipLaunchKernelGGL(lz_scale4_kernel<B>, dim3(grid_for(n / 4)), dim3(NT), 0, s, w, qnext, basis_row,
                       (const double*)(st.beta + k), (const int*)st.flag, n);
  else
  hipLaunchKernelGGL(lz_scale_kernel<B>, dim3(grid_for(n)), dim3(NT), 0, s, w, qnext, basis_row,
                     (const double*)(st.beta + k), (const int*)st.flag, n);
  return hipGetLastError();
}

#define INST_LZ(B)                                                                                              \
  template hipError_t launch_lanczos_b<B>(float*, const float*, const B*, int, LanczosDev, int, int64_t, hipStream_t); \
  template hipError_t launch_lanczos_cgs<B>(float*, const B*, int, LanczosDev, int, bool, int, int64_t, hipStream_t);  \
  template hipError_t launch_lanczos_normalise<B>(const float*, float*, B*, LanczosDev, int, double, int64_t, hipStream_t);
INST_LZ(float)
INST_LZ(bf16_t)

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
