// Counter-based SplitMix64 generator (Steele, Lea and Flood, OOPSLA 2014) and
// the synthetic inputs drawn from it.
//
// The i-th output (0-based) of stream (seed, stream) is
//     mix(key + (i + 1) * 0x9E3779B97F4A7C15),  key = seed * 2^16 + stream,
// with the SplitMix64 finaliser mix.  Derived variates, all formed in fp64:
//   uniform  u = ((h >> 11) + 0.5) * 2^-53
//   normal   element i: sqrt(-2 ln u(2i)) * cos(2 pi u(2i+1))
//   sign     -1 when the top bit of output i is set
//   token    uniform: ((h >> 32) * V) >> 32;  Zipf: first rank k with cdf[k] >= u
#include "kernels.h"

namespace fdh {

namespace {

constexpr uint64_t GAMMA = 0x9E3779B97F4A7C15ull;

__device__ inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
__device__ inline uint64_t sm64(uint64_t seed, uint64_t stream, uint64_t i) {
  return mix64((seed << 16) + stream + (i + 1) * GAMMA);
}
__device__ inline double unif(uint64_t h) { return ((double)(h >> 11) + 0.5) * 0x1.0p-53; }
__device__ inline double normal_at(uint64_t seed, uint64_t stream, uint64_t i) {
  const double u1 = unif(sm64(seed, stream, 2 * i));
  const double u2 = unif(sm64(seed, stream, 2 * i + 1));
  return sqrt(-2.0 * log(u1)) * cos(2.0 * 3.141592653589793 * u2);
}

template <typename T>
__global__ void init_range_kernel(T* theta, int64_t off, int64_t n, int kind, uint64_t seed, double stdv) {
  for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < n; j += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = off + j;
    float x;
    if (kind == 0) x = (float)(stdv * normal_at(seed, STREAM_PARAMS, (uint64_t)i));
    else if (kind == 1) x = 1.0f;
    else x = 0.0f;
    stf(theta, i, x);
  }
}

__global__ void tokens_uniform_kernel(int32_t* tok, int64_t n, uint64_t seed, uint32_t V) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const uint64_t h = sm64(seed, STREAM_TOKENS, (uint64_t)i);
    tok[i] = (int32_t)(((h >> 32) * (uint64_t)V) >> 32);
  }
}

__global__ void tokens_zipf_kernel(int32_t* tok, int64_t n, uint64_t seed, const double* cdf, int V) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const double u = unif(sm64(seed, STREAM_TOKENS, (uint64_t)i));
    int lo = 0, hi = V;  // first index with cdf[idx] >= u
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (cdf[mid] < u) lo = mid + 1; else hi = mid;
    }
    tok[i] = lo < V ? lo : V - 1;
  }
}

__global__ void rademacher_kernel(float* out, int64_t n, uint64_t seed, double inv_norm_div) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const uint64_t h = sm64(seed, STREAM_PROBE, (uint64_t)i);
    const double s = (h >> 63) ? -1.0 : 1.0;
    out[i] = (float)(s / inv_norm_div);
  }
}

__global__ void gaussian_kernel(float* out, double* partial, int64_t n, uint64_t seed) {
  __shared__ double sh[4];
  double acc = 0.0;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const double g = normal_at(seed, STREAM_GAUSS, (uint64_t)i);
    acc += g * g;
  }
  acc = block_sum<256>(acc, sh);
  if (threadIdx.x == 0) partial[blockIdx.x] = acc;
}

__global__ void gaussian_write_kernel(float* out, const double* partial, int nb, int64_t n, uint64_t seed) {
  __shared__ double nrm;
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int b = 0; b < nb; ++b) s += partial[b];
    nrm = sqrt(s);
  }
  __syncthreads();
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    out[i] = (float)(normal_at(seed, STREAM_GAUSS, (uint64_t)i) / nrm);
}

unsigned grid_for(int64_t n) {
  int64_t g = (n + 255) / 256;
  if (g > 65536) g = 65536;
  if (g < 1) g = 1;
  return (unsigned)g;
}

}  // namespace

template <typename T>
hipError_t launch_init_range(T* theta, int64_t off, int64_t n, int kind, uint64_t seed, double stdv, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(init_range_kernel<T>, dim3(grid_for(n)), dim3(256), 0, s, theta, off, n, kind, seed, stdv);
  return hipGetLastError();
}
template hipError_t launch_init_range<float>(float*, int64_t, int64_t, int, uint64_t, double, hipStream_t);
template hipError_t launch_init_range<bf16_t>(bf16_t*, int64_t, int64_t, int, uint64_t, double, hipStream_t);

hipError_t launch_tokens_uniform(int32_t* tok, int64_t n, uint64_t seed, int V, hipStream_t s) {
  hipLaunchKernelGGL(tokens_uniform_kernel, dim3(grid_for(n)), dim3(256), 0, s, tok, n, seed, (uint32_t)V);
  return hipGetLastError();
}
hipError_t launch_tokens_zipf(int32_t* tok, int64_t n, uint64_t seed, const double* cdf, int V, hipStream_t s) {
  hipLaunchKernelGGL(tokens_zipf_kernel, dim3(grid_for(n)), dim3(256), 0, s, tok, n, seed, cdf, V);
  return hipGetLastError();
}
hipError_t launch_rademacher(float* out, int64_t n, uint64_t seed, hipStream_t s) {
  hipLaunchKernelGGL(rademacher_kernel, dim3(grid_for(n)), dim3(256), 0, s, out, n, seed, sqrt((double)n));
  return hipGetLastError();
}
// partial must hold 1024 doubles
hipError_t launch_gaussian_unit(float* out, double* partial, int64_t n, uint64_t seed, hipStream_t s) {
  const int nb = 1024;
  hipLaunchKernelGGL(gaussian_kernel, dim3(nb), dim3(256), 0, s, out, partial, n, seed);
  hipLaunchKernelGGL(gaussian_write_kernel, dim3(grid_for(n)), dim3(256), 0, s, out, partial, nb, n, seed);
  return hipGetLastError();
}

}  // namespace fdh
