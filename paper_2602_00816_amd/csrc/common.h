// Internal helpers shared by the HIP kernels and the host engine.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>
#include <cstddef>

namespace fdh {

// ---------------------------------------------------------------------------
// bfloat16 stored as uint16_t bit patterns
// ---------------------------------------------------------------------------
typedef uint16_t bf16_t;

__host__ __device__ inline float bf16_to_f32(bf16_t h) {
  union { uint32_t u; float f; } c;
  c.u = ((uint32_t)h) << 16;
  return c.f;
}

// round-to-nearest-even float32 -> bfloat16 (NaN kept quiet): the compiler's
// conversion, one v_cvt_pk_bf16_f32 per pair of values on gfx950
__host__ __device__ inline bf16_t f32_to_bf16(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

template <typename T> struct OpType;
template <> struct OpType<float> {
  __device__ static inline float load(const float* p, int64_t i) { return p[i]; }
  __device__ static inline void store(float* p, int64_t i, float x) { p[i] = x; }
};
template <> struct OpType<bf16_t> {
  __device__ static inline float load(const bf16_t* p, int64_t i) { return bf16_to_f32(p[i]); }
  __device__ static inline void store(bf16_t* p, int64_t i, float x) { p[i] = f32_to_bf16(x); }
};

template <typename T> __device__ inline float ldf(const T* p, int64_t i) { return OpType<T>::load(p, i); }
template <typename T> __device__ inline void stf(T* p, int64_t i, float x) { OpType<T>::store(p, i, x); }

// ---------------------------------------------------------------------------
// wavefront / block reductions (64-wide wavefronts)
// ---------------------------------------------------------------------------
__device__ inline double wave_sum(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}
__device__ inline float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}
__device__ inline double wave_max(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmax(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ inline float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}

// Sum over a block of NT threads (NT multiple of 64, <= 1024); every thread
// receives the result.  The order of additions is fixed, so the result is
// reproducible.  `sh` must hold NT/64 doubles.
template <int NT>
__device__ inline double block_sum(double x, double* sh) {
  x = wave_sum(x);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) sh[w] = x;
  __syncthreads();
  double t = 0.0;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) t += sh[i];
  return t;
}
template <int NT>
__device__ inline double block_max(double x, double* sh) {
  x = wave_max(x);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) sh[w] = x;
  __syncthreads();
  double t = sh[0];
#pragma unroll
  for (int i = 1; i < NT / 64; ++i) t = fmax(t, sh[i]);
  return t;
}

inline unsigned ceil_div(int64_t a, int64_t b) { return (unsigned)((a + b - 1) / b); }

}  // namespace fdh
