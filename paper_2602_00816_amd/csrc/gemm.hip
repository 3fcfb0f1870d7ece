// Batched MFMA GEMM for gfx950.
//
// One workgroup of 256 threads (4 wavefronts of 64) computes a 128x128 tile of
// C.  Each wavefront owns a 64x64 quarter as 2x2 blocks of 32x32 MFMA
// accumulators (v_mfma_f32_32x32x16_bf16 for bf16 operands,
// v_mfma_f32_32x32x2_f32 for fp32 operands).  A and B tiles are staged in LDS
// in K-contiguous rows; operands that are stored MN-major in HBM are
// transposed while being written to LDS, so the MFMA fragment reads are always
// single 16-byte (bf16) or 4-byte (fp32) LDS reads.  Global loads are 16-byte
// vectors, prefetched into registers one K-tile ahead.
#include "gemm.h"

namespace fdh {

namespace {

constexpr int BM = 128, BN = 128, NT = 256;

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;

template <typename T> struct Tr;
template <> struct Tr<bf16_t> {
  static constexpr int KT = 32;   // K per LDS tile
  static constexpr int VEC = 8;   // elements per 16-byte vector
  static constexpr int PAD = 8;   // LDS row padding (elements)
};
template <> struct Tr<float> {
  static constexpr int KT = 16;
  static constexpr int VEC = 4;
  static constexpr int PAD = 4;
};

struct alignas(16) Vec16 { uint32_t w[4]; };

__device__ inline int64_t batch_off(int z, int inner_count, int64_t s_outer, int64_t s_inner, int div) {
  return (int64_t)(z / inner_count) * s_outer + (int64_t)((z % inner_count) / div) * s_inner;
}

// Load the VEC-element vector number `i` (0..1) of this thread for a tile
// starting at (row0, k0).  Returns zeros outside [0,rows) x [0,K).
template <typename T, bool KMAJ>
__device__ inline Vec16 load_vec(const T* base, int64_t s_row, int64_t s_k, int rows, int K,
                                 int row0, int k0, int vid) {
  constexpr int KT = Tr<T>::KT, VEC = Tr<T>::VEC;
  Vec16 v = {{0u, 0u, 0u, 0u}};
  if (KMAJ) {
    const int r = vid / (KT / VEC);
    const int kk = (vid % (KT / VEC)) * VEC;
    const int gr = row0 + r, gk = k0 + kk;
    if (gr < rows && gk < K) v = *reinterpret_cast<const Vec16*>(base + (int64_t)gr * s_row + gk);
  } else {
    const int kk = vid / (BM / VEC);
    const int r = (vid % (BM / VEC)) * VEC;
    const int gr = row0 + r, gk = k0 + kk;
    if (gr < rows && gk < K) v = *reinterpret_cast<const Vec16*>(base + (int64_t)gk * s_k + gr);
  }
  return v;
}

template <typename T, bool KMAJ>
__device__ inline void store_vec(T* s, const Vec16& v, int vid) {
  constexpr int KT = Tr<T>::KT, VEC = Tr<T>::VEC, LD = KT + Tr<T>::PAD;
  if (KMAJ) {
    const int r = vid / (KT / VEC);
    const int kk = (vid % (KT / VEC)) * VEC;
    *reinterpret_cast<Vec16*>(s + r * LD + kk) = v;
  } else {
    const int kk = vid / (BM / VEC);
    const int r = (vid % (BM / VEC)) * VEC;
    const T* e = reinterpret_cast<const T*>(&v);
#pragma unroll
    for (int j = 0; j < VEC; ++j) s[(r + j) * LD + kk] = e[j];
  }
}

template <typename T>
__device__ inline void mma_tile(const T* sA, const T* sB, f32x16_t (&acc)[2][2], int wm, int wn, int lane);

template <>
__device__ inline void mma_tile<bf16_t>(const bf16_t* sA, const bf16_t* sB, f32x16_t (&acc)[2][2],
                                        int wm, int wn, int lane) {
  constexpr int LD = Tr<bf16_t>::KT + Tr<bf16_t>::PAD;
#pragma unroll
  for (int kk = 0; kk < Tr<bf16_t>::KT; kk += 16) {
    bf16x8_t af[2], bfr[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const bf16_t* pa = sA + (wm * 64 + i * 32 + (lane & 31)) * LD + kk + 8 * (lane >> 5);
      af[i] = *reinterpret_cast<const bf16x8_t*>(pa);
      const bf16_t* pb = sB + (wn * 64 + i * 32 + (lane & 31)) * LD + kk + 8 * (lane >> 5);
      bfr[i] = *reinterpret_cast<const bf16x8_t*>(pb);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
  }
}

template <>
__device__ inline void mma_tile<float>(const float* sA, const float* sB, f32x16_t (&acc)[2][2],
                                       int wm, int wn, int lane) {
  constexpr int LD = Tr<float>::KT + Tr<float>::PAD;
#pragma unroll
  for (int kk = 0; kk < Tr<float>::KT; kk += 2) {
    float af[2], bfr[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      af[i] = sA[(wm * 64 + i * 32 + (lane & 31)) * LD + kk + (lane >> 5)];
      bfr[i] = sB[(wn * 64 + i * 32 + (lane & 31)) * LD + kk + (lane >> 5)];
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i], bfr[j], acc[i][j], 0, 0, 0);
  }
}

template <typename T, bool AK, bool BKM>
__global__ __launch_bounds__(NT) void gemm_kernel(GemmArgs a) {
  constexpr int KT = Tr<T>::KT, LD = KT + Tr<T>::PAD;
  __shared__ __attribute__((aligned(16))) T sA[BM * LD];
  __shared__ __attribute__((aligned(16))) T sB[BN * LD];

  const int z = blockIdx.z;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  if (a.causal == CAUSAL_SKIP_UPPER && n0 > m0 + BM - 1) return;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  int kmin = 0, kmax = a.K;
  if (a.causal == CAUSAL_K_LE_M) kmax = min(a.K, m0 + BM);
  if (a.causal == CAUSAL_K_GE_M) kmin = (min(m0, a.K) / KT) * KT;

  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  for (int p = 0; p < a.npairs; ++p) {
    const GemmOperand& A = a.A[p];
    const GemmOperand& B = a.B[p];
    const T* pa = reinterpret_cast<const T*>(A.ptr) + batch_off(z, a.inner_count, A.s_outer, A.s_inner, A.inner_div);
    const T* pb = reinterpret_cast<const T*>(B.ptr) + batch_off(z, a.inner_count, B.s_outer, B.s_inner, B.inner_div);
    Vec16 ra[2], rb[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      ra[i] = load_vec<T, AK>(pa, A.s_row, A.s_k, a.M, kmax, m0, kmin, tid + i * NT);
      rb[i] = load_vec<T, BKM>(pb, B.s_row, B.s_k, a.N, kmax, n0, kmin, tid + i * NT);
    }
    for (int k0 = kmin; k0 < kmax; k0 += KT) {
      __syncthreads();
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        store_vec<T, AK>(sA, ra[i], tid + i * NT);
        store_vec<T, BKM>(sB, rb[i], tid + i * NT);
      }
      __syncthreads();
      if (k0 + KT < kmax) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          ra[i] = load_vec<T, AK>(pa, A.s_row, A.s_k, a.M, kmax, m0, k0 + KT, tid + i * NT);
          rb[i] = load_vec<T, BKM>(pb, B.s_row, B.s_k, a.N, kmax, n0, k0 + KT, tid + i * NT);
        }
      }
      mma_tile<T>(sA, sB, acc, wm, wn, lane);
    }
  }

  // epilogue
  const int64_t coff = batch_off(z, a.inner_count, a.c_outer, a.c_inner, a.c_div);
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wn * 64 + j * 32 + (lane & 31);
      if (col >= a.N) continue;
      float badd = 0.f;
      if (a.bias_theta) badd += a.bias_theta_scale * ldf(reinterpret_cast<const T*>(a.bias_theta), col);
      if (a.bias_v) badd += a.bias_v_scale * a.bias_v[col];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 64 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        if (row >= a.M) continue;
        const int64_t idx = coff + (int64_t)row * a.ldc + col;
        float x = a.alpha * acc[i][j][r] + badd;
        if (a.out_type == OUT_F32) {
          float* C = reinterpret_cast<float*>(a.C);
          if (a.resid) x += a.resid[idx];
          if (a.beta != 0.f) x += a.beta * C[idx];
          C[idx] = x;
        } else {
          stf(reinterpret_cast<T*>(a.C), idx, x);
        }
      }
    }
}

}  // namespace

template <typename T>
const char* gemm_check(const GemmArgs& a) {
  constexpr int VEC = Tr<T>::VEC;
  if (a.M < 0 || a.N < 0 || a.K < 0 || a.nbatch < 1 || a.inner_count < 1) return "gemm: bad sizes";
  if (a.npairs < 1 || a.npairs > 2) return "gemm: npairs must be 1 or 2";
  if (a.K % VEC) return "gemm: K must be a multiple of the 16-byte vector width";
  if (!a.C) return "gemm: null C";
  if (a.beta != 0.f && a.out_type != OUT_F32) return "gemm: beta needs fp32 output";
  if (a.resid && a.out_type != OUT_F32) return "gemm: residual needs fp32 output";
  bool ak = a.A[0].s_k == 1, bk = a.B[0].s_k == 1;
  for (int p = 0; p < a.npairs; ++p) {
    const GemmOperand* ops[2] = {&a.A[p], &a.B[p]};
    const int rows[2] = {a.M, a.N};
    for (int q = 0; q < 2; ++q) {
      const GemmOperand& o = *ops[q];
      if (!o.ptr) return "gemm: null operand";
      if ((reinterpret_cast<uintptr_t>(o.ptr) & 15) != 0) return "gemm: operand not 16-byte aligned";
      if (o.inner_div < 1) return "gemm: inner_div < 1";
      if (o.s_outer % VEC || o.s_inner % VEC) return "gemm: batch strides must be vector multiples";
      const bool km = o.s_k == 1;
      if (km == (q == 0 ? !ak : !bk)) return "gemm: pairs must share operand layouts";
      if (km) {
        if (o.s_row % VEC) return "gemm: row stride must be a vector multiple";
      } else {
        if (o.s_row != 1) return "gemm: one of s_row, s_k must be 1";
        if (o.s_k % VEC) return "gemm: k stride must be a vector multiple";
        if (rows[q] % VEC) return "gemm: MN-major operand rows must be a vector multiple";
      }
    }
  }
  if (a.causal != CAUSAL_NONE && a.M > a.N && a.causal == CAUSAL_SKIP_UPPER) return "gemm: causal skip needs M <= N";
  return nullptr;
}

template <typename T>
hipError_t gemm(const GemmArgs& a, hipStream_t stream) {
  if (a.M == 0 || a.N == 0) return hipSuccess;
  dim3 grid(ceil_div(a.N, BN), ceil_div(a.M, BM), a.nbatch);
  const bool ak = a.A[0].s_k == 1, bk = a.B[0].s_k == 1;
  if (ak && bk) hipLaunchKernelGGL((gemm_kernel<T, true, true>), grid, dim3(NT), 0, stream, a);
  else if (ak && !bk) hipLaunchKernelGGL((gemm_kernel<T, true, false>), grid, dim3(NT), 0, stream, a);
  else if (!ak && bk) hipLaunchKernelGGL((gemm_kernel<T, false, true>), grid, dim3(NT), 0, stream, a);
  else hipLaunchKernelGGL((gemm_kernel<T, false, false>), grid, dim3(NT), 0, stream, a);
  return hipGetLastError();
}

template hipError_t gemm<float>(const GemmArgs&, hipStream_t);
template hipError_t gemm<bf16_t>(const GemmArgs&, hipStream_t);
template const char* gemm_check<float>(const GemmArgs&);
template const char* gemm_check<bf16_t>(const GemmArgs&);

}  // namespace fdh
