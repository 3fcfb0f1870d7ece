// Batched MFMA GEMM for gfx950:  C[z] = alpha * sum_p A_p[z] B_p[z]^T (+ epilogue).
//
// Two kernels:
//  * gemm_kernel  - 128x128 workgroup tile, 4 wavefronts of 64x64 (2x2 blocks
//    of 32x32 MFMA accumulators), fp32 (v_mfma_f32_32x32x2_f32) or bf16
//    (v_mfma_f32_32x32x16_bf16) operands; used for fp32 and for small bf16
//    problems.
//  * gemm_bf16_big - bf16 only, 256x256 (8 wavefronts) or 256x128 (4
//    wavefronts) workgroup tiles; every wavefront owns 128x64 as 4x2 blocks of
//    32x32, so one A fragment read from LDS feeds two MFMAs and one B fragment
//    four.  K tile 64, LDS double-buffered, one barrier per K tile.
// Both stage A and B in LDS as K-contiguous rows.  Operands stored MN-major in
// HBM are transposed on their way into LDS, so the MFMA fragment reads are
// always single 16-byte LDS reads.  Global loads are 16-byte vectors,
// prefetched into registers one K tile ahead.
#include "gemm.h"

#include <type_traits>

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

// ===========================================================================
// 128x128 kernel
// ===========================================================================
// Load the 16-byte vector number `vid` of a tile starting at (row0, k0).
// Returns zeros outside [0,rows) x [0,K).
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
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
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
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(bfr[j], af[i], acc[i][j], 0, 0, 0);
  }
}

// shared epilogue: accumulator block (i, j) of a wavefront whose 32x32 block
// origin is (rb, cb).  Every MFMA takes the B fragment as its first operand, so
// the block holds C^T in the MFMA output layout: lane l owns row rb + (l & 31)
// of C and, for g = 0..3, the four consecutive columns cb + 8g + 4(l >> 5) + 0..3
// (accumulator elements 4g..4g+3).  Each such quad is stored, and the residual
// or previous C loaded, as one vector where the addresses are aligned.
// four consecutive outputs at C[idx..idx+3], 16-byte (fp32) or 8-byte (bf16)
// aligned: one vector store, with the residual and previous C read as vectors
template <typename T>
__device__ inline void store_quad(const GemmArgs& a, const float (&x)[4], int64_t idx) {
  if (a.out_type == OUT_F32) {
    float* C = reinterpret_cast<float*>(a.C);
    float4 v = make_float4(x[0], x[1], x[2], x[3]);
    if (a.resid) {
      const float4 r = *reinterpret_cast<const float4*>(a.resid + idx);
      v.x += r.x; v.y += r.y; v.z += r.z; v.w += r.w;
    }
    if (a.beta != 0.f) {
      const float4 c = *reinterpret_cast<const float4*>(C + idx);
      v.x += a.beta * c.x; v.y += a.beta * c.y; v.z += a.beta * c.z; v.w += a.beta * c.w;
    }
    *reinterpret_cast<float4*>(C + idx) = v;
  } else {
    T* C = reinterpret_cast<T*>(a.C);
    if constexpr (sizeof(T) == 2) {
      uint2 u;
      u.x = (uint32_t)f32_to_bf16(x[0]) | ((uint32_t)f32_to_bf16(x[1]) << 16);
      u.y = (uint32_t)f32_to_bf16(x[2]) | ((uint32_t)f32_to_bf16(x[3]) << 16);
      *reinterpret_cast<uint2*>(C + idx) = u;
    } else {
      *reinterpret_cast<float4*>(C + idx) = make_float4(x[0], x[1], x[2], x[3]);
    }
  }
}

template <typename T>
__device__ inline void store_block(const GemmArgs& a, const f32x16_t& acc, int64_t coff, int rb, int cb, int lane) {
  const int row = rb + (lane & 31);
  if (row >= a.M) return;
  const int64_t rbase = coff + (int64_t)row * a.ldc;
  // vector path: row starts and column quads aligned for 16-byte (fp32) or
  // 8-byte (bf16) accesses
  const size_t ob = a.out_type == OUT_F32 ? 4 : sizeof(T);
  const bool aligned = a.ldc % 4 == 0 && coff % 4 == 0 && (uintptr_t)a.C % (4 * ob) == 0 &&
                       (!a.resid || (uintptr_t)a.resid % 16 == 0);
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int col0 = cb + 8 * g + 4 * (lane >> 5);
    if (col0 >= a.N) continue;
    float x[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int col = min(col0 + r, a.N - 1);
      float badd = 0.f;
      if (a.bias_theta) badd += a.bias_theta_scale * ldf(reinterpret_cast<const T*>(a.bias_theta), col);
      if (a.bias_v) badd += a.bias_v_scale * a.bias_v[col];
      x[r] = a.alpha * acc[4 * g + r] + badd;
    }
    if (aligned && col0 + 3 < a.N) {
      store_quad<T>(a, x, rbase + col0);
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (col0 + r >= a.N) break;
        const int64_t idx = rbase + col0 + r;
        float y = x[r];
        if (a.out_type == OUT_F32) {
          float* C = reinterpret_cast<float*>(a.C);
          if (a.resid) y += a.resid[idx];
          if (a.beta != 0.f) y += a.beta * C[idx];
          C[idx] = y;
        } else {
          stf(reinterpret_cast<T*>(a.C), idx, y);
        }
      }
    }
  }
}

// LDS-staged epilogue of one 32x32 block: the wavefront writes its block
// (scaled by alpha) to its own staging area of 32 rows x 36 floats, then reads
// it back so that lane l holds row 8k + (l >> 3), columns 4(l & 7) + 0..3:
// every global access then covers eight rows of 128 contiguous bytes.  The
// caller guarantees the staging area is not in use by the main loop any more.
constexpr int STG_LD = 36;
constexpr int STG_FLOATS = 32 * STG_LD;
// four staging areas fit one ring stage of the DMA kernels (256 x 32 + 128 x 32 bf16 at the smallest)
static_assert(4 * STG_FLOATS * 4 <= (256 + 128) * 32 * 2, "staging areas exceed a ring stage");
static_assert(4 * STG_FLOATS * 4 <= (256 + 256) * 32 * 2, "four blocks of staging exceed a 256 x 256 ring stage");
// (the eight-wavefront kernel gives each pair of wavefronts one 256 x 256 stage, two blocks each)

__device__ inline void wave_lds_order() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <typename T>
__device__ inline void store_block_lds(const GemmArgs& a, const f32x16_t& acc, int64_t coff, int rb, int cb, int lane,
                                       float* stg) {
  {
    const int wr = lane & 31, wh = lane >> 5;
#pragma unroll
    for (int g = 0; g < 4; ++g)
      *reinterpret_cast<float4*>(stg + wr * STG_LD + 8 * g + 4 * wh) =
          make_float4(a.alpha * acc[4 * g], a.alpha * acc[4 * g + 1], a.alpha * acc[4 * g + 2], a.alpha * acc[4 * g + 3]);
  }
  wave_lds_order();
  const int c4 = 4 * (lane & 7);
  const int col0 = cb + c4;
  float badd[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int col = min(col0 + r, a.N - 1);
    if (a.bias_theta) badd[r] += a.bias_theta_scale * ldf(reinterpret_cast<const T*>(a.bias_theta), col);
    if (a.bias_v) badd[r] += a.bias_v_scale * a.bias_v[col];
  }
  const size_t ob = a.out_type == OUT_F32 ? 4 : sizeof(T);
  const bool aligned = a.ldc % 4 == 0 && coff % 4 == 0 && (uintptr_t)a.C % (4 * ob) == 0 &&
                       (!a.resid || (uintptr_t)a.resid % 16 == 0);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int lr = 8 * k + (lane >> 3);
    const float4 v = *reinterpret_cast<const float4*>(stg + lr * STG_LD + c4);
    const int row = rb + lr;
    if (row >= a.M || col0 >= a.N) continue;
    const float x[4] = {v.x + badd[0], v.y + badd[1], v.z + badd[2], v.w + badd[3]};
    const int64_t base = coff + (int64_t)row * a.ldc + col0;
    if (aligned && col0 + 3 < a.N) {
      store_quad<T>(a, x, base);
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (col0 + r >= a.N) break;
        float y = x[r];
        if (a.out_type == OUT_F32) {
          float* C = reinterpret_cast<float*>(a.C);
          if (a.resid) y += a.resid[base + r];
          if (a.beta != 0.f) y += a.beta * C[base + r];
          C[base + r] = y;
        } else {
          stf(reinterpret_cast<T*>(a.C), base + r, y);
        }
      }
    }
  }
  wave_lds_order();   // the next block's writes come after these reads
}

// LDS-staged epilogue of NB 32x32 blocks of one wavefront (blocks (rb, cb[j]),
// j < NB) in one round: all NB are written to the wavefront's staging area
// (NB x 32 rows x 36 floats), then every lane reads its 4 NB quads, issues
// every global read the epilogue needs (residual, previous C) before any
// store, and stores.  One round has the latency of one block where the
// one-block form pays it NB times (a wavefront that is alone on its SIMD has
// nothing else to hide it with).  Global accesses cover eight rows of
// 128 contiguous bytes, as in store_block_lds.
template <typename T, int NB>
__device__ inline void store_blocks_lds(const GemmArgs& a, const f32x16_t (&acc)[NB], int64_t coff, int rb,
                                        const int (&cb)[NB], int lane, float* stg) {
  {
    const int wr = lane & 31, wh = lane >> 5;
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<float4*>(stg + j * STG_FLOATS + wr * STG_LD + 8 * g + 4 * wh) =
            make_float4(a.alpha * acc[j][4 * g], a.alpha * acc[j][4 * g + 1], a.alpha * acc[j][4 * g + 2],
                        a.alpha * acc[j][4 * g + 3]);
  }
  wave_lds_order();
  const int c4 = 4 * (lane & 7);
  float4 v[NB][4];
#pragma unroll
  for (int j = 0; j < NB; ++j)
#pragma unroll
    for (int k = 0; k < 4; ++k) v[j][k] = *reinterpret_cast<const float4*>(stg + j * STG_FLOATS + (8 * k + (lane >> 3)) * STG_LD + c4);
  wave_lds_order();   // the next round's writes come after these reads
  const size_t ob = a.out_type == OUT_F32 ? 4 : sizeof(T);
  const bool aligned = a.ldc % 4 == 0 && coff % 4 == 0 && (uintptr_t)a.C % (4 * ob) == 0 &&
                       (!a.resid || (uintptr_t)a.resid % 16 == 0);
  const bool full = aligned && rb + 32 <= a.M && cb[NB - 1] + 32 <= a.N;
  if (full && a.out_type == OUT_F32 && !a.bias_theta && !a.bias_v) {
    // the common case of the residual stream and the weight gradients: all
    // reads first, then all stores
    float* C = reinterpret_cast<float*>(a.C);
    float4 r[NB][4];
    const bool rd = a.resid != nullptr, bt = a.beta != 0.f;
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int64_t idx = coff + (int64_t)(rb + 8 * k + (lane >> 3)) * a.ldc + cb[j] + c4;
        float4 t = make_float4(0.f, 0.f, 0.f, 0.f);
        if (rd) t = *reinterpret_cast<const float4*>(a.resid + idx);
        if (bt) {
          const float4 c = *reinterpret_cast<const float4*>(C + idx);
          t.x += a.beta * c.x; t.y += a.beta * c.y; t.z += a.beta * c.z; t.w += a.beta * c.w;
        }
        r[j][k] = t;
      }
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int64_t idx = coff + (int64_t)(rb + 8 * k + (lane >> 3)) * a.ldc + cb[j] + c4;
        *reinterpret_cast<float4*>(C + idx) =
            make_float4(v[j][k].x + r[j][k].x, v[j][k].y + r[j][k].y, v[j][k].z + r[j][k].z, v[j][k].w + r[j][k].w);
      }
    return;
  }
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int col0 = cb[j] + c4;
    float badd[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int col = min(col0 + q, a.N - 1);
      if (a.bias_theta) badd[q] += a.bias_theta_scale * ldf(reinterpret_cast<const T*>(a.bias_theta), col);
      if (a.bias_v) badd[q] += a.bias_v_scale * a.bias_v[col];
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int row = rb + 8 * k + (lane >> 3);
      if (row >= a.M || col0 >= a.N) continue;
      const float x[4] = {v[j][k].x + badd[0], v[j][k].y + badd[1], v[j][k].z + badd[2], v[j][k].w + badd[3]};
      const int64_t base = coff + (int64_t)row * a.ldc + col0;
      if (aligned && col0 + 3 < a.N) {
        store_quad<T>(a, x, base);
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (col0 + q >= a.N) break;
          float y = x[q];
          if (a.out_type == OUT_F32) {
            float* C = reinterpret_cast<float*>(a.C);
            if (a.resid) y += a.resid[base + q];
            if (a.beta != 0.f) y += a.beta * C[base + q];
            C[base + q] = y;
          } else {
            stf(reinterpret_cast<T*>(a.C), base + q, y);
          }
        }
      }
    }
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

  const int64_t coff = batch_off(z, a.inner_count, a.c_outer, a.c_inner, a.c_div);
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
      store_block<T>(a, acc[i][j], coff, m0 + wm * 64 + i * 32, n0 + wn * 64 + j * 32, lane);
}

// ===========================================================================
// bf16 kernel with large tiles: BM x BN workgroup tile, WM x WN wavefronts,
// each wavefront 128 x 64 (4 x 2 blocks of 32x32).
// ===========================================================================
// LDS holds each tile row as 64 bf16 = 128 bytes (8 chunks of 16 bytes) with
// the chunk index XOR-swizzled by bits 0-2 and 3-5 of the row: the 16-byte
// MFMA fragment reads (8 consecutive rows, one chunk), the 16-byte K-major
// stores (one row, 8 chunks) and the 8-byte transposed stores (rows 8 apart,
// one chunk) all spread over the 32 LDS banks.
constexpr int KT2 = 64, LD2 = KT2;
__device__ inline int swz(int row, int chunk) { return row * LD2 + ((chunk ^ (row & 7) ^ ((row >> 3) & 7)) << 3); }
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// One R x KT2 tile.  K-major: R*8 vectors of 8 consecutive k; MN-major:
// 2R bundles of 4 consecutive k x 8 consecutive rows, transposed in registers
// into 8-byte LDS rows.  NTH threads share the work.
template <int R, bool KMAJ, int NTH>
struct TileLoader {
  static constexpr int UNITS = KMAJ ? R * 8 : 2 * R;        // vectors or bundles
  static constexpr int PER = (UNITS + NTH - 1) / NTH;       // units per thread
  static constexpr int NV = KMAJ ? PER : 4 * PER;           // 16-byte registers per thread
  u32x4 v[NV];

  __device__ inline void load(const bf16_t* base, int64_t s_row, int64_t s_k, int rows, int kmax, int row0, int k0,
                              int tid) {
#pragma clang loop unroll(full)
    for (int u = 0; u < PER; ++u) {
      const int id = tid + u * NTH;
      if (KMAJ) {
        const int r = id >> 3, kk = (id & 7) * 8;
        const int gr = row0 + r, gk = k0 + kk;
        u32x4 x = {0u, 0u, 0u, 0u};
        if (id < UNITS && gr < rows && gk < kmax) x = *reinterpret_cast<const u32x4*>(base + (int64_t)gr * s_row + gk);
        v[u] = x;
      } else {
        const int rg = id % (R / 8), kq = id / (R / 8);
        const int gr = row0 + rg * 8;
#pragma clang loop unroll(full)
        for (int j = 0; j < 4; ++j) {
          const int gk = k0 + kq * 4 + j;
          u32x4 x = {0u, 0u, 0u, 0u};
          if (id < UNITS && gr < rows && gk < kmax) x = *reinterpret_cast<const u32x4*>(base + (int64_t)gk * s_k + gr);
          v[4 * u + j] = x;
        }
      }
    }
  }

  __device__ inline void store(bf16_t* s, int tid) const {
#pragma clang loop unroll(full)
    for (int u = 0; u < PER; ++u) {
      const int id = tid + u * NTH;
      if (id >= UNITS) continue;
      if (KMAJ) {
        const int r = id >> 3, kk = (id & 7) * 8;
        *reinterpret_cast<u32x4*>(s + swz(r, kk >> 3)) = v[u];
      } else {
        const int rg = id % (R / 8), kq = id / (R / 8);
        const u32x4* w = &v[4 * u];
#pragma clang loop unroll(full)
        for (int q = 0; q < 4; ++q) {
          // rows 2q (low halves) and 2q+1 (high halves) of the four k vectors
          uint2 ev, od;
          ev.x = (w[0][q] & 0xFFFFu) | (w[1][q] << 16);
          ev.y = (w[2][q] & 0xFFFFu) | (w[3][q] << 16);
          od.x = (w[0][q] >> 16) | (w[1][q] & 0xFFFF0000u);
          od.y = (w[2][q] >> 16) | (w[3][q] & 0xFFFF0000u);
          *reinterpret_cast<uint2*>(s + swz(rg * 8 + 2 * q, kq >> 1) + (kq & 1) * 4) = ev;
          *reinterpret_cast<uint2*>(s + swz(rg * 8 + 2 * q + 1, kq >> 1) + (kq & 1) * 4) = od;
        }
      }
    }
  }
};

template <int BM_, int BN_, int WM, int WN, bool AK, bool BKM>
__global__ __launch_bounds__(64 * WM * WN) void gemm_bf16_big(GemmArgs a) {
  constexpr int NTH = 64 * WM * WN;
  constexpr int IM = BM_ / (32 * WM), JN = BN_ / (32 * WN);
  __shared__ __attribute__((aligned(16))) bf16_t sA[2][BM_ * LD2];
  __shared__ __attribute__((aligned(16))) bf16_t sB[2][BN_ * LD2];

  // XCD-aware tile order.  Workgroups are handed to the 8 XCDs round-robin
  // in launch order; renumber so that each XCD receives one contiguous run of
  // tiles, and walk tiles in groups of 8 row panels so that the workgroups
  // resident on one XCD share A and B panels in that XCD's L2.
  const int gx = gridDim.x, gy = gridDim.y;
  const int nb = gx * gy * gridDim.z;
  int lin = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
  const int per = nb / 8;
  if (lin < per * 8) lin = (lin % 8) * per + lin / 8;
  const int tiles = gx * gy;
  const int z = lin / tiles;
  const int tl = lin % tiles;
  constexpr int GM = 8;
  const int gsize = GM * gx;
  const int first_m = (tl / gsize) * GM;
  const int gm_rows = min(gy - first_m, GM);
  const int tm = first_m + (tl % gsize) % gm_rows;
  const int tn = (tl % gsize) / gm_rows;
  const int m0 = tm * BM_, n0 = tn * BN_;
  if (a.causal == CAUSAL_SKIP_UPPER && n0 > m0 + BM_ - 1) return;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  int kmin = 0, kmax = a.K;
  if (a.causal == CAUSAL_K_LE_M) kmax = min(a.K, m0 + BM_);
  if (a.causal == CAUSAL_K_GE_M) kmin = (min(m0, a.K) / KT2) * KT2;

  f32x16_t acc[IM][JN];
#pragma clang loop unroll(full)
  for (int i = 0; i < IM; ++i)
#pragma clang loop unroll(full)
    for (int j = 0; j < JN; ++j)
#pragma clang loop unroll(full)
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  TileLoader<BM_, AK, NTH> la;
  TileLoader<BN_, BKM, NTH> lb;
  const int nkt = (kmax > kmin) ? (kmax - kmin + KT2 - 1) / KT2 : 0;
  const int total = nkt * a.npairs;

  // operand bases of both pairs (pair p covers K tiles p*nkt .. p*nkt + nkt - 1)
  const bf16_t* pa0 = reinterpret_cast<const bf16_t*>(a.A[0].ptr) +
                      batch_off(z, a.inner_count, a.A[0].s_outer, a.A[0].s_inner, a.A[0].inner_div);
  const bf16_t* pb0 = reinterpret_cast<const bf16_t*>(a.B[0].ptr) +
                      batch_off(z, a.inner_count, a.B[0].s_outer, a.B[0].s_inner, a.B[0].inner_div);
  const bf16_t* pa1 = pa0;
  const bf16_t* pb1 = pb0;
  if (a.npairs > 1) {
    pa1 = reinterpret_cast<const bf16_t*>(a.A[1].ptr) +
          batch_off(z, a.inner_count, a.A[1].s_outer, a.A[1].s_inner, a.A[1].inner_div);
    pb1 = reinterpret_cast<const bf16_t*>(a.B[1].ptr) +
          batch_off(z, a.inner_count, a.B[1].s_outer, a.B[1].s_inner, a.B[1].inner_div);
  }
  const int64_t asr0 = a.A[0].s_row, ask0 = a.A[0].s_k, bsr0 = a.B[0].s_row, bsk0 = a.B[0].s_k;
  const int64_t asr1 = a.A[1].s_row, ask1 = a.A[1].s_k, bsr1 = a.B[1].s_row, bsk1 = a.B[1].s_k;

  if (total > 0) {
    la.load(pa0, asr0, ask0, a.M, kmax, m0, kmin, tid);
    lb.load(pb0, bsr0, bsk0, a.N, kmax, n0, kmin, tid);
    la.store(sA[0], tid);
    lb.store(sB[0], tid);
    __syncthreads();
  }
  for (int t = 0; t < total; ++t) {
    const int cur = t & 1;
    if (t + 1 < total) {
      const int t1 = t + 1;
      const bool second = t1 >= nkt;
      const int k0 = kmin + (second ? t1 - nkt : t1) * KT2;
      la.load(second ? pa1 : pa0, second ? asr1 : asr0, second ? ask1 : ask0, a.M, kmax, m0, k0, tid);
      lb.load(second ? pb1 : pb0, second ? bsr1 : bsr0, second ? bsk1 : bsk0, a.N, kmax, n0, k0, tid);
    }
    const bf16_t* cA = sA[cur];
    const bf16_t* cB = sB[cur];
#pragma clang loop unroll(full)
    for (int kk = 0; kk < KT2; kk += 16) {
      bf16x8_t af[IM], bfr[JN];
#pragma clang loop unroll(full)
      for (int i = 0; i < IM; ++i)
        af[i] = *reinterpret_cast<const bf16x8_t*>(cA + swz(wm * (BM_ / WM) + i * 32 + (lane & 31), (kk >> 3) + (lane >> 5)));
#pragma clang loop unroll(full)
      for (int j = 0; j < JN; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8_t*>(cB + swz(wn * (BN_ / WN) + j * 32 + (lane & 31), (kk >> 3) + (lane >> 5)));
#pragma clang loop unroll(full)
      for (int i = 0; i < IM; ++i)
#pragma clang loop unroll(full)
        for (int j = 0; j < JN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
    }
    if (t + 1 < total) {
      la.store(sA[cur ^ 1], tid);
      lb.store(sB[cur ^ 1], tid);
    }
    __syncthreads();
  }

  const int64_t coff = batch_off(z, a.inner_count, a.c_outer, a.c_inner, a.c_div);
#pragma clang loop unroll(full)
  for (int i = 0; i < IM; ++i)
#pragma clang loop unroll(full)
    for (int j = 0; j < JN; ++j)
      store_block<bf16_t>(a, acc[i][j], coff, m0 + wm * (BM_ / WM) + i * 32, n0 + wn * (BN_ / WN) + j * 32, lane);
}

// ===========================================================================
// bf16 kernel fed by direct global->LDS loads (global_load_lds_dwordx4).
//
// A 4-stage LDS ring of K = 32 slices: the loads for slice t + 3 are issued
// right after the barrier that opens slice t, so three slices (~3 us of MFMA
// work) cover the memory latency, and no VGPR holds prefetched data.  Each
// load instruction writes 64 lanes x 16 bytes contiguously in LDS (lane l at
// +16 l), so the global address of each lane is chosen to match the swizzled
// LDS position it lands in.
//   K-major tile (rows x 32 k): 64-byte rows, 16-byte chunk c of row r stored
//     at chunk c ^ ((r >> 2) & 3); MFMA fragments are single 16-byte reads.
//   MN-major tile (32 k x rows): rows of `rows` elements along m/n, chunk c of
//     k-row k stored at c ^ (4 (k & 3)); MFMA fragments are two transposing
//     reads (ds_read_b64_tr_b16), each giving a lane 4 consecutive k of its
//     m/n column.
// The LDS has 64 banks of 4 bytes and serves a 16-byte read for 16 lanes, an
// 8-byte read for 32 lanes per clock; in both layouts those lanes hit 64
// distinct banks, and the DMA writes are contiguous.
// Requires K, kmin, kmax multiples of 32; rows past M/N are clamped to valid
// memory (they only feed discarded outputs).
// ===========================================================================
constexpr int KT3 = 32, NS3 = 4;
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16_t;
typedef __attribute__((address_space(3))) void lds_void_t;

__device__ inline int kswz(int row, int c) { return row * KT3 + ((c ^ ((row >> 2) & 3)) << 3); }        // elements
template <int R>
__device__ inline int mswz(int k, int m) { return k * R + ((((m >> 3) ^ (4 * (k & 3)))) << 3) + (m & 7); }  // elements

// issue this wave's DMA instructions for one operand tile
template <int R, bool KMAJ, int NW>
__device__ inline void dma_tile(bf16_t* lds_tile, const bf16_t* base, int64_t s_row, int64_t s_k, int rows, int row0,
                                int k0, int wave, int lane) {
  constexpr int NI = R * KT3 * 2 / 1024;  // 1 KB instructions per tile
#pragma clang loop unroll(full)
  for (int u = 0; u < NI / NW; ++u) {
    const int q = wave + u * NW;
    const bf16_t* g;
    if (KMAJ) {
      const int r = q * 16 + (lane >> 2);                       // 16 rows of 64 B per instruction
      const int c = (lane & 3) ^ ((r >> 2) & 3);
      const int gr = min(row0 + r, rows - 1);
      g = base + (int64_t)gr * s_row + k0 + 8 * c;
    } else {
      constexpr int RPI = 1024 / (R * 2);                       // k-rows per instruction
      constexpr int CPR = R / 8;                                // chunks per k-row
      const int k = q * RPI + lane / CPR;
      const int c = (lane % CPR) ^ (4 * (k & 3));
      const int gm = min(row0 + 8 * c, rows - 8);
      g = base + (int64_t)(k0 + k) * s_k + gm;
    }
    // Issued as inline assembly so that the compiler does not track it: its
    // own tracking cannot tell the ring stages apart and would wait for every
    // outstanding load before each LDS read.  Completion is waited for
    // explicitly (wait_vm) before the barrier that publishes a stage.
    const uint32_t ldsaddr = (uint32_t)(uintptr_t)(lds_void_t*)(lds_tile + q * 512);
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off"
        :
        : "s"(__builtin_amdgcn_readfirstlane(ldsaddr)), "v"(g)
        : "memory", "m0");
  }
}

template <int R, bool KMAJ>
__device__ inline bf16x8_t frag(const bf16_t* t, int r0, int kk, int lane) {
  if (KMAJ) {
    return *reinterpret_cast<const bf16x8_t*>(t + kswz(r0 + (lane & 31), (kk >> 3) + (lane >> 5)));
  } else {
    const int g = lane >> 4, r = lane & 15;
    const int mb = r0 + 16 * (g & 1) + 4 * (r & 3);
    const int kb = kk + 8 * (g >> 1) + (r >> 2);
    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(t + mswz<R>(kb, mb)));
    const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(t + mswz<R>(kb + 4, mb)));
    typedef short v8i16 __attribute__((ext_vector_type(8)));
    const v8i16 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8_t, v);
  }
}

template <int N>
__device__ inline void wait_vm() {
  // s_waitcnt with vmcnt = N (bits 3:0 and 15:14), expcnt and lgkmcnt left at their maxima
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

#ifndef FDH_DMA_STAGES
#define FDH_DMA_STAGES 4
#endif
template <int BN_, int WN, bool AK, bool BKM>
__global__ __launch_bounds__(64 * 2 * WN) void gemm_bf16_dma(GemmArgs a) {
  constexpr int BM_ = 256, WM = 2, NW = WM * WN;
  // ring depth: 4 stages, or 5 for 256-wide tiles when built with FDH_DMA_STAGES=5
  constexpr int NS = (BN_ == 256 && FDH_DMA_STAGES == 5) ? 5 : 4;
  constexpr int WTN = BN_ / WN;                 // wavefront tile: 128 x WTN
  constexpr int IM = 4, JN = WTN / 32;
  constexpr int ASZ = BM_ * KT3, BSZ = BN_ * KT3;              // elements per stage
  constexpr int PERT = (BM_ + BN_) * KT3 * 2 / 1024 / NW;      // DMA instructions per wave per tile
  // one LDS object per stage: with compile-time stage indices the compiler
  // waits, before an LDS read, only for the DMA into that same stage
  __shared__ __attribute__((aligned(1024))) bf16_t st0[ASZ + BSZ];
  __shared__ __attribute__((aligned(1024))) bf16_t st1[ASZ + BSZ];
  __shared__ __attribute__((aligned(1024))) bf16_t st2[ASZ + BSZ];
  __shared__ __attribute__((aligned(1024))) bf16_t st3[ASZ + BSZ];
  __shared__ __attribute__((aligned(1024))) bf16_t st4[NS == 5 ? ASZ + BSZ : 8];

  const int gx = gridDim.x, gy = gridDim.y;
  const int nb = gx * gy * gridDim.z;
  int lin = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
  const int per = nb / 8;
  if (lin < per * 8) lin = (lin % 8) * per + lin / 8;
  const int tiles = gx * gy;
  const int z = lin / tiles;
  const int tl = lin % tiles;
  constexpr int GM = 8;
  const int gsize = GM * gx;
  const int first_m = (tl / gsize) * GM;
  const int gm_rows = min(gy - first_m, GM);
  const int tm = first_m + (tl % gsize) % gm_rows;
  const int tn = (tl % gsize) / gm_rows;
  const int m0 = tm * BM_, n0 = tn * BN_;
  if (a.causal == CAUSAL_SKIP_UPPER && n0 > m0 + BM_ - 1) return;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;

  int kmin = 0, kmax = a.K;
  if (a.causal == CAUSAL_K_LE_M) kmax = min(a.K, m0 + BM_);
  if (a.causal == CAUSAL_K_GE_M) kmin = (min(m0, a.K) / KT3) * KT3;
  const int nkt = (kmax > kmin) ? (kmax - kmin) / KT3 : 0;
  const int total = nkt * a.npairs;

  const bf16_t* pa[2];
  const bf16_t* pb[2];
#pragma clang loop unroll(full)
  for (int p = 0; p < 2; ++p) {
    const int pp = p < a.npairs ? p : 0;
    pa[p] = reinterpret_cast<const bf16_t*>(a.A[pp].ptr) +
            batch_off(z, a.inner_count, a.A[pp].s_outer, a.A[pp].s_inner, a.A[pp].inner_div);
    pb[p] = reinterpret_cast<const bf16_t*>(a.B[pp].ptr) +
            batch_off(z, a.inner_count, a.B[pp].s_outer, a.B[pp].s_inner, a.B[pp].inner_div);
  }

  auto stage = [&](auto s) -> bf16_t* {
    constexpr int S = decltype(s)::value;
    if constexpr (S == 0) return st0;
    else if constexpr (S == 1) return st1;
    else if constexpr (S == 2) return st2;
    else if constexpr (S == 3) return st3;
    else return st4;
  };
  auto issue = [&](int t, bf16_t* st) {
    const int p = t >= nkt ? 1 : 0;
    const int k0 = kmin + (t - p * nkt) * KT3;
    dma_tile<BM_, AK, NW>(st, p ? pa[1] : pa[0], a.A[p].s_row, a.A[p].s_k, a.M, m0, k0, wave, lane);
    dma_tile<BN_, BKM, NW>(st + ASZ, p ? pb[1] : pb[0], a.B[p].s_row, a.B[p].s_k, a.N, n0, k0, wave, lane);
  };

  f32x16_t acc[IM][JN];
#pragma clang loop unroll(full)
  for (int i = 0; i < IM; ++i)
#pragma clang loop unroll(full)
    for (int j = 0; j < JN; ++j)
#pragma clang loop unroll(full)
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // one K slice on stage S (compile time): wait for this wave's loads of the
  // slice (later slices stay in flight), barrier, refill the stage freed by
  // the previous slice, then 2 x IM x JN MFMAs
  auto step = [&](auto s, int t) {
    constexpr int S = decltype(s)::value;
    const int ahead = min(NS - 2, total - 1 - t);
    if (ahead >= 3) wait_vm<3 * PERT>();
    else if (ahead == 2) wait_vm<2 * PERT>();
    else if (ahead == 1) wait_vm<PERT>();
    else wait_vm<0>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");  // keep the stage's LDS reads after the barrier
    if (t + NS - 1 < total) issue(t + NS - 1, stage(std::integral_constant<int, (S + NS - 1) % NS>{}));
    const bf16_t* cA = stage(s);
    const bf16_t* cB = cA + ASZ;
#pragma clang loop unroll(full)
    for (int kk = 0; kk < KT3; kk += 16) {
      bf16x8_t af[IM], bfr[JN];
#pragma clang loop unroll(full)
      for (int i = 0; i < IM; ++i) af[i] = frag<BM_, AK>(cA, wm * 128 + i * 32, kk, lane);
#pragma clang loop unroll(full)
      for (int j = 0; j < JN; ++j) bfr[j] = frag<BN_, BKM>(cB, wn * WTN + j * 32, kk, lane);
#pragma clang loop unroll(full)
      for (int i = 0; i < IM; ++i)
#pragma clang loop unroll(full)
        for (int j = 0; j < JN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
    }
  };

  if (total > 0) issue(0, st0);
  if (total > 1) issue(1, st1);
  if (total > 2) issue(2, st2);
  if (NS == 5 && total > 3) issue(3, st3);
  for (int t0 = 0; t0 < total; t0 += NS) {
    step(std::integral_constant<int, 0>{}, t0);
    if (t0 + 1 < total) step(std::integral_constant<int, 1>{}, t0 + 1);
    if (t0 + 2 < total) step(std::integral_constant<int, 2>{}, t0 + 2);
    if (t0 + 3 < total) step(std::integral_constant<int, 3>{}, t0 + 3);
    if constexpr (NS == 5)
      if (t0 + 4 < total) step(std::integral_constant<int, 4>{}, t0 + 4);
  }

  const int64_t coff = batch_off(z, a.inner_count, a.c_outer, a.c_inner, a.c_div);
  // stage the output through the ring once every wavefront is done with it:
  // two blocks per round, 2 x 32 x 36 floats per wavefront
  wait_vm<0>();
  __syncthreads();
  const int wv = threadIdx.x >> 6;
  if constexpr (JN == 2 && NW == 8) {
    float* stg = reinterpret_cast<float*>(wv < 2 ? st0 : wv < 4 ? st1 : wv < 6 ? st2 : st3) + (wv & 1) * 2 * STG_FLOATS;
    const int cbs[2] = {n0 + wn * WTN, n0 + wn * WTN + 32};
#pragma clang loop unroll(full)
    for (int i = 0; i < IM; ++i) store_blocks_lds<bf16_t, 2>(a, acc[i], coff, m0 + wm * 128 + i * 32, cbs, lane, stg);
  } else {
    float* stg = reinterpret_cast<float*>(wv < 4 ? st0 : st1) + (wv & 3) * STG_FLOATS;
#pragma clang loop unroll(full)
    for (int i = 0; i < IM; ++i)
#pragma clang loop unroll(full)
      for (int j = 0; j < JN; ++j)
        store_block_lds<bf16_t>(a, acc[i][j], coff, m0 + wm * 128 + i * 32, n0 + wn * WTN + j * 32, lane, stg);
  }
}

// ===========================================================================
// bf16 GEMM, 256 x 256 block tile, four wavefronts of 128 x 128 each (one per
// SIMD; WN = 2), on the same DMA-fed LDS ring and LDS layouts as
// gemm_bf16_dma.  With 128 x 128 per wavefront every fragment read from LDS
// feeds four MFMAs instead of two or three, which halves LDS read traffic per
// FLOP.  WN = 4 runs the same schedule on eight wavefronts of 128 x 64 (two
// per SIMD, 220 registers), which trades LDS reads for a second wavefront to
// hide latency and a shorter prologue and epilogue per tile.  A wavefront
// keeps two fragment register sets and its instruction order is fixed by
// scheduling barriers: a K slice is two half slices of 16 k; while the 16
// MFMAs of one half run, the fragments of the next half are read.  The loads
// of a slice are spread over two half slices, one load per two MFMAs: A's
// into the stage freed at the ring barrier (three slices ahead), B's during
// the next half slice (then two and a half slices ahead), which keeps the
// load queue shorter than issuing all eight at once (measured 1.5-3% faster
// on the 1.3B layer shapes, same bits).  Loads past the last slice reload the
// last slice into the free stage (never read), so every slice issues the same
// number of loads and the vmcnt waits are constants.
// ===========================================================================
// One 256 x 256 output tile of the product a: tile lin of a gx x gy tile grid
// (times a.nbatch).
template <bool AK, bool BKM, int WN>
__device__ __forceinline__ void w4_tile(const GemmArgs& a, int gx, int gy, int lin) {
  // WN = 2: four wavefronts of 128 x 128; WN = 4: eight of 128 x 64
  constexpr int BM_ = 256, BN_ = 256, NW = 2 * WN, IM = 4, JN = 8 / WN, WTN = BN_ / WN;
  constexpr int ASZ = BM_ * KT3, BSZ = BN_ * KT3;
  constexpr int NU = BM_ * KT3 * 2 / 1024 / NW;   // 1 KB loads per operand per wavefront per slice
  constexpr int PERT = 2 * NU;                    // loads per wavefront per slice
  __shared__ __attribute__((aligned(1024))) bf16_t st0[ASZ + BSZ];
  __shared__ __attribute__((aligned(1024))) bf16_t st1[ASZ + BSZ];
  __shared__ __attribute__((aligned(1024))) bf16_t st2[ASZ + BSZ];
  __shared__ __attribute__((aligned(1024))) bf16_t st3[ASZ + BSZ];

  const int tiles = gx * gy;
  const int z = lin / tiles;
  const int tl = lin % tiles;
  // tiles run down GM tile rows before the next column (with the XCD
  // renumbering, each XCD's 32 concurrent tiles then share 4 A and 8 B
  // operand blocks); 4 measured 0.35% faster per HVP than 8 and 16 slower
  constexpr int GM = 4;
  const int gsize = GM * gx;
  const int first_m = (tl / gsize) * GM;
  const int gm_rows = min(gy - first_m, GM);
  const int tm = first_m + (tl % gsize) % gm_rows;
  const int tn = (tl % gsize) / gm_rows;
  const int m0 = tm * BM_, n0 = tn * BN_;
  if (a.causal == CAUSAL_SKIP_UPPER && n0 > m0 + BM_ - 1) return;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;

  int kmin = 0, kmax = a.K;
  if (a.causal == CAUSAL_K_LE_M) kmax = min(a.K, m0 + BM_);
  if (a.causal == CAUSAL_K_GE_M) kmin = (min(m0, a.K) / KT3) * KT3;
  const int nkt = (kmax > kmin) ? (kmax - kmin) / KT3 : 0;
  const int total = nkt * a.npairs;

  // per-lane source offsets (elements) of this wavefront's loads, both pairs
  const bf16_t* baseA[2];
  const bf16_t* baseB[2];
  int64_t offA[2][NU], offB[2][NU], skA[2], skB[2];
#pragma clang loop unroll(full)
  for (int p = 0; p < 2; ++p) {
    const int pp = p < a.npairs ? p : 0;
    const GemmOperand& A = a.A[pp];
    const GemmOperand& B = a.B[pp];
    baseA[p] = reinterpret_cast<const bf16_t*>(A.ptr) + batch_off(z, a.inner_count, A.s_outer, A.s_inner, A.inner_div);
    baseB[p] = reinterpret_cast<const bf16_t*>(B.ptr) + batch_off(z, a.inner_count, B.s_outer, B.s_inner, B.inner_div);
    skA[p] = AK ? 1 : A.s_k;
    skB[p] = BKM ? 1 : B.s_k;
#pragma clang loop unroll(full)
    for (int u = 0; u < NU; ++u) {
      const int q = wave + u * NW;
      // K-major: 16 rows of 64 B per load; MN-major: 2 k-rows of 512 B per load
      const int r = q * 16 + (lane >> 2), ck = (lane & 3) ^ ((r >> 2) & 3);
      const int k = q * 2 + (lane >> 5), cm = (lane & 31) ^ (4 * (k & 3));
      offA[p][u] = AK ? (int64_t)min(m0 + r, a.M - 1) * A.s_row + 8 * ck
                      : (int64_t)k * A.s_k + min(m0 + 8 * cm, a.M - 8);
      offB[p][u] = BKM ? (int64_t)min(n0 + r, a.N - 1) * B.s_row + 8 * ck
                       : (int64_t)k * B.s_k + min(n0 + 8 * cm, a.N - 8);
    }
  }

  auto stage = [&](auto s) -> bf16_t* {
    constexpr int S = decltype(s)::value & 3;
    if constexpr (S == 0) return st0;
    else if constexpr (S == 1) return st1;
    else if constexpr (S == 2) return st2;
    else return st3;
  };
  // load u (0..2 NU-1) of slice t (clamped to the last slice) into stage st
  auto dma = [&](bf16_t* st, int t, int u) {
    t = min(t, total - 1);
    const int p = t >= nkt ? 1 : 0;
    const int64_t k0 = kmin + (t - p * nkt) * KT3;
    const bool isA = u < NU;
    const int uu = isA ? u : u - NU;
    const int q = wave + uu * NW;
    const bf16_t* g = isA ? (p ? baseA[1] + offA[1][uu] + k0 * skA[1] : baseA[0] + offA[0][uu] + k0 * skA[0])
                          : (p ? baseB[1] + offB[1][uu] + k0 * skB[1] : baseB[0] + offB[0][uu] + k0 * skB[0]);
    // LDS byte address: stage base (a link-time constant) + wave-uniform offset
    const uint32_t ldsaddr = (uint32_t)(uintptr_t)(lds_void_t*)st + (uint32_t)(((isA ? 0 : ASZ) + q * 512) * 2);
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off"
        :
        : "s"(ldsaddr), "v"(g)
        : "memory", "m0");
  };

  f32x16_t acc[IM][JN];
#pragma clang loop unroll(full)
  for (int i = 0; i < IM; ++i)
#pragma clang loop unroll(full)
    for (int j = 0; j < JN; ++j)
#pragma clang loop unroll(full)
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  bf16x8_t f0[IM + JN], f1[IM + JN];   // fragments of half slices (k 0..15, k 16..31)
  auto rd = [&](bf16x8_t& f, const bf16_t* st, int x, int kk) {
    if (x < IM) f = frag<BM_, AK>(st, wm * 128 + x * 32, kk, lane);
    else f = frag<BN_, BKM>(st + ASZ, wn * WTN + (x - IM) * 32, kk, lane);
  };
  auto mma = [&](const bf16x8_t (&f)[IM + JN], int e) {
    const int i = e / JN, j = e % JN;
    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[IM + j], f[i], acc[i][j], 0, 0, 0);
  };

  auto step = [&](auto s, int t) {
    constexpr int S = decltype(s)::value;
    const bf16_t* cur = stage(s);
    bf16_t* fill2 = stage(std::integral_constant<int, S + 2>{});
    // half slice 0 on f0 (read during the previous slice); read half 1 into
    // f1; issue B's loads of slice t + 2 into the stage freed at the previous
    // barrier (A's went out during the previous half slice)
#pragma clang loop unroll(full)
    for (int x = 0; x < IM + JN; ++x) {
      rd(f1[x], cur, x, 16);
      if ((x & 1) && x / 2 < NU) dma(fill2, t + 2, NU + x / 2);
#pragma clang loop unroll(full)
      for (int e = x * IM * JN / (IM + JN); e < (x + 1) * IM * JN / (IM + JN); ++e) mma(f0, e);
      __builtin_amdgcn_sched_barrier(0);
    }
    // own loads of slice t + 1 done (the 8 issued since are slice t + 2's),
    // then everyone's; stage S - 1 is free
    wait_vm<PERT>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    bf16_t* nxt_fill = stage(std::integral_constant<int, S + 3>{});
    const bf16_t* nxt = stage(std::integral_constant<int, S + 1>{});
    // half slice 1 on f1; A's loads of slice t + 3 into stage S - 1; read half 0 of slice t + 1 into f0
#pragma clang loop unroll(full)
    for (int x = 0; x < IM + JN; ++x) {
      if ((x & 1) && x / 2 < NU) dma(nxt_fill, t + 3, x / 2);
      rd(f0[x], nxt, x, 0);
#pragma clang loop unroll(full)
      for (int e = x * IM * JN / (IM + JN); e < (x + 1) * IM * JN / (IM + JN); ++e) mma(f1, e);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  if (total > 0) {
    // slices 0 and 1, and A's loads of slice 2 (B's go out in the first step)
#pragma clang loop unroll(full)
    for (int u = 0; u < 2 * NU; ++u) dma(st0, 0, u);
#pragma clang loop unroll(full)
    for (int u = 0; u < 2 * NU; ++u) dma(st1, 1, u);
#pragma clang loop unroll(full)
    for (int u = 0; u < NU; ++u) dma(st2, 2, u);
    wait_vm<PERT + NU>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
#pragma clang loop unroll(full)
    for (int x = 0; x < IM + JN; ++x) rd(f0[x], st0, x, 0);
    for (int t0 = 0; t0 < total; t0 += NS3) {
      step(std::integral_constant<int, 0>{}, t0);
      if (t0 + 1 < total) step(std::integral_constant<int, 1>{}, t0 + 1);
      if (t0 + 2 < total) step(std::integral_constant<int, 2>{}, t0 + 2);
      if (t0 + 3 < total) step(std::integral_constant<int, 3>{}, t0 + 3);
    }
    wait_vm<0>();   // no load may land in LDS after the workgroup ends
  }

  const int64_t coff = batch_off(z, a.inner_count, a.c_outer, a.c_inner, a.c_div);
  // stage the output through the ring once every wavefront is done with it:
  // four wavefronts: wavefront w uses stage w (4 x 32 x 36 floats = 18 KB of
  // its 32 KB); eight: wavefronts 2s and 2s + 1 share stage s, 2 blocks each
  __syncthreads();
  if constexpr (WN == 2) {
    float* stg = reinterpret_cast<float*>(wave == 0 ? st0 : wave == 1 ? st1 : wave == 2 ? st2 : st3);
    const int cbs[4] = {n0 + wn * 128, n0 + wn * 128 + 32, n0 + wn * 128 + 64, n0 + wn * 128 + 96};
#pragma clang loop unroll(full)
    for (int i = 0; i < IM; ++i)
      store_blocks_lds<bf16_t, 4>(a, acc[i], coff, m0 + wm * 128 + i * 32, cbs, lane, stg);
  } else {
    float* stg = reinterpret_cast<float*>(wave < 2 ? st0 : wave < 4 ? st1 : wave < 6 ? st2 : st3) +
                 (wave & 1) * 2 * STG_FLOATS;
    const int cbs[2] = {n0 + wn * WTN, n0 + wn * WTN + 32};
#pragma clang loop unroll(full)
    for (int i = 0; i < IM; ++i)
      store_blocks_lds<bf16_t, 2>(a, acc[i], coff, m0 + wm * 128 + i * 32, cbs, lane, stg);
  }
}

// Workgroup ids are dealt to the 8 XCDs in turn; renumber them so that each
// XCD takes a contiguous run of tiles (neighbouring tiles share operand rows
// and columns in that XCD's L2).
__device__ inline int xcd_order(int lin, int nb) {
  const int per = nb / 8;
  return lin < per * 8 ? (lin % 8) * per + lin / 8 : lin;
}

template <bool AK, bool BKM, int WN = 2>
__global__ __launch_bounds__(64 * 2 * WN) void gemm_bf16_w4(GemmArgs a) {
  const int gx = gridDim.x, gy = gridDim.y;
  w4_tile<AK, BKM, WN>(a, gx, gy, xcd_order(blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z), gx * gy * gridDim.z));
}

// Two independent products in one grid (one-dimensional, the n0 tiles of a0,
// batch entries included, then those of a1): the tiles of a1 take the compute
// units that a grid of a0 alone would leave idle in its last wave.  Each product is renumbered on
// its own, so that every XCD takes an eighth of each (renumbering the joint
// grid would give a0 to some XCDs and a1 to the others).
template <bool AK, bool BKM, int WN = 2>
__global__ __launch_bounds__(64 * 2 * WN) void gemm_bf16_w4_pair(GemmArgs a0, GemmArgs a1, int n0) {
  const int b = blockIdx.x;
  if (b < n0) w4_tile<AK, BKM, WN>(a0, (a0.N + 255) / 256, (a0.M + 255) / 256, xcd_order(b, n0));
  else w4_tile<AK, BKM, WN>(a1, (a1.N + 255) / 256, (a1.M + 255) / 256, xcd_order(b - n0, gridDim.x - n0));
}

// ===========================================================================
// As gemm_bf16_w4 with K slices of 64 in a two-stage ring (2 x 64 KB).  A
// K-major row of a slice is one whole 128-byte line, so each DMA load moves 8
// full lines (half as many L1/L2 requests per byte as 64-byte row pieces),
// and there is one barrier per 64 k.  A slice is four half slices of 16 k
// read and multiplied in a two-register-set rotation; after the third, each
// wavefront waits for its own LDS reads of the stage and for its loads of the
// next slice, then the barrier frees the stage for the slice after next.
// K-major LDS layout: row r of a slice is 8 chunks of 16 B, logical chunk c at
// c ^ ((r >> 1) & 7) (16 lanes reading 16 consecutive rows hit 64 banks).
// ===========================================================================
constexpr int KT4 = 64;
typedef int i32x4_t __attribute__((ext_vector_type(4)));
__device__ inline int kswz64(int row, int c) { return row * KT4 + ((c ^ ((row >> 1) & 7)) << 3); }   // elements

template <int R, bool KMAJ>
__device__ inline bf16x8_t frag64(const bf16_t* t, int r0, int kk, int lane) {
  if (KMAJ) return *reinterpret_cast<const bf16x8_t*>(t + kswz64(r0 + (lane & 31), (kk >> 3) + (lane >> 5)));
  return frag<R, false>(t, r0, kk, lane);
}

template <bool AK, bool BKM>
__global__ __launch_bounds__(256) void gemm_bf16_w4k64(GemmArgs a) {
  constexpr int BM_ = 256, BN_ = 256, NW = 4, IM = 4, JN = 4;
  constexpr int ASZ = BM_ * KT4, BSZ = BN_ * KT4;
  constexpr int NU = BM_ * KT4 * 2 / 1024 / NW;   // 1 KB loads per operand per wavefront per slice (8)
  constexpr int SSZ = ASZ + BSZ;                  // elements per stage
  __shared__ __attribute__((aligned(1024))) bf16_t ring[2 * SSZ];

  const int gx = gridDim.x, gy = gridDim.y;
  const int nb = gx * gy * gridDim.z;
  int lin = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
  const int per = nb / 8;
  if (lin < per * 8) lin = (lin % 8) * per + lin / 8;
  const int tiles = gx * gy;
  const int z = lin / tiles;
  const int tl = lin % tiles;
  constexpr int GM = 8;
  const int gsize = GM * gx;
  const int first_m = (tl / gsize) * GM;
  const int gm_rows = min(gy - first_m, GM);
  const int tm = first_m + (tl % gsize) % gm_rows;
  const int tn = (tl % gsize) / gm_rows;
  const int m0 = tm * BM_, n0 = tn * BN_;
  if (a.causal == CAUSAL_SKIP_UPPER && n0 > m0 + BM_ - 1) return;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  int kmin = 0, kmax = a.K;
  if (a.causal == CAUSAL_K_LE_M) kmax = min(a.K, m0 + BM_);
  if (a.causal == CAUSAL_K_GE_M) kmin = (min(m0, a.K) / KT4) * KT4;
  const int nkt = (kmax > kmin) ? (kmax - kmin) / KT4 : 0;
  const int total = nkt * a.npairs;

  // Loads go through buffer resources whose base is the slice origin of the
  // tile (row m0 / n0, column k0), so each lane keeps one small 32-bit byte
  // offset per load for the whole K loop.  Both pairs share these offsets:
  // their operands have equal strides (checked on the host).
  const bf16_t* baseA[2];
  const bf16_t* baseB[2];
#pragma clang loop unroll(full)
  for (int p = 0; p < 2; ++p) {
    const int pp = p < a.npairs ? p : 0;
    const GemmOperand& A = a.A[pp];
    const GemmOperand& B = a.B[pp];
    baseA[p] = reinterpret_cast<const bf16_t*>(A.ptr) + batch_off(z, a.inner_count, A.s_outer, A.s_inner, A.inner_div) +
               (AK ? (int64_t)m0 * A.s_row : (int64_t)m0);
    baseB[p] = reinterpret_cast<const bf16_t*>(B.ptr) + batch_off(z, a.inner_count, B.s_outer, B.s_inner, B.inner_div) +
               (BKM ? (int64_t)n0 * B.s_row : (int64_t)n0);
  }
  const int64_t skA = AK ? 1 : a.A[0].s_k, skB = BKM ? 1 : a.B[0].s_k;
  uint32_t voA[NU], voB[NU];
#pragma clang loop unroll(full)
  for (int u = 0; u < NU; ++u) {
    const int q = wave + u * NW;
    // K-major: 8 rows of 128 B per load; MN-major: 2 k-rows of 512 B per load
    const int r = q * 8 + (lane >> 3), ck = (lane & 7) ^ ((r >> 1) & 7);
    const int k = q * 2 + (lane >> 5), cm = (lane & 31) ^ (4 * (k & 3));
    voA[u] = 2u * (uint32_t)(AK ? (int64_t)(min(m0 + r, a.M - 1) - m0) * a.A[0].s_row + 8 * ck
                                : (int64_t)k * a.A[0].s_k + (min(m0 + 8 * cm, a.M - 8) - m0));
    voB[u] = 2u * (uint32_t)(BKM ? (int64_t)(min(n0 + r, a.N - 1) - n0) * a.B[0].s_row + 8 * ck
                                 : (int64_t)k * a.B[0].s_k + (min(n0 + 8 * cm, a.N - 8) - n0));
  }

  // raw buffer resource: base, stride 0, no range limit, 32-bit data format
  auto rsrc = [](const bf16_t* base) {
    const uint64_t b = (uint64_t)(uintptr_t)base;
    return i32x4_t{(int)(uint32_t)b, (int)((b >> 32) & 0xffffu), -1, 0x00020000};
  };
  // load u (0..2 NU-1) of slice t (clamped to the last slice) into stage st
  auto dma = [&](bf16_t* st, int t, int u) {
    t = min(t, total - 1);
    const int p = t >= nkt ? 1 : 0;
    const int64_t k0 = kmin + (t - p * nkt) * KT4;
    const bool isA = u < NU;
    const int uu = isA ? u : u - NU;
    const int q = wave + uu * NW;
    const i32x4_t rs = isA ? rsrc((p ? baseA[1] : baseA[0]) + k0 * skA) : rsrc((p ? baseB[1] : baseB[0]) + k0 * skB);
    const uint32_t vo = isA ? voA[uu] : voB[uu];
    const uint32_t ldsaddr = (uint32_t)(uintptr_t)(lds_void_t*)st + (uint32_t)(((isA ? 0 : ASZ) + q * 512) * 2);
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen lds"
        :
        : "s"(ldsaddr), "v"(vo), "s"(rs)
        : "memory", "m0");
  };

  f32x16_t acc[IM][JN];
#pragma clang loop unroll(full)
  for (int i = 0; i < IM; ++i)
#pragma clang loop unroll(full)
    for (int j = 0; j < JN; ++j)
#pragma clang loop unroll(full)
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  bf16x8_t f0[IM + JN], f1[IM + JN];
  auto rd = [&](bf16x8_t& f, const bf16_t* st, int x, int kk) {
    if (x < IM) f = frag64<BM_, AK>(st, wm * 128 + x * 32, kk, lane);
    else f = frag64<BN_, BKM>(st + ASZ, wn * 128 + (x - IM) * 32, kk, lane);
  };
  auto mma = [&](const bf16x8_t (&f)[IM + JN], int e) {
    const int i = e / JN, j = e % JN;
    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[IM + j], f[i], acc[i][j], 0, 0, 0);
  };
  // one half slice: MFMAs on `use`, fragments of the next half slice into `load`
  auto half = [&](const bf16x8_t (&use)[IM + JN], bf16x8_t (&load)[IM + JN], const bf16_t* st, int kk) {
#pragma clang loop unroll(full)
    for (int x = 0; x < IM + JN; ++x) {
      rd(load[x], st, x, kk);
      mma(use, 2 * x);
      mma(use, 2 * x + 1);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // The stage is a run-time choice (one slice per loop trip, no branches
  // inside the trip, so the accumulators stay in place across iterations).
  auto step = [&](int t) {
    bf16_t* cur = ring + (t & 1) * SSZ;
    const bf16_t* nxt = ring + ((t + 1) & 1) * SSZ;
    half(f0, f1, cur, 16);
    half(f1, f0, cur, 32);
    half(f0, f1, cur, 48);
    // this wavefront's reads of the stage and its loads of slice t + 1 are
    // complete; after the barrier everyone's are, and the stage is free
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
#pragma clang loop unroll(full)
    for (int x = 0; x < IM + JN; ++x) {
      dma(cur, t + 2, 2 * x);
      dma(cur, t + 2, 2 * x + 1);
      rd(f0[x], nxt, x, 0);
      mma(f1, 2 * x);
      mma(f1, 2 * x + 1);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  if (total > 0) {
#pragma clang loop unroll(full)
    for (int u = 0; u < 2 * NU; ++u) dma(ring, 0, u);
#pragma clang loop unroll(full)
    for (int u = 0; u < 2 * NU; ++u) dma(ring + SSZ, 1, u);
    wait_vm<2 * NU>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
#pragma clang loop unroll(full)
    for (int x = 0; x < IM + JN; ++x) rd(f0[x], ring, x, 0);
#pragma clang loop unroll(disable)
    for (int t = 0; t < total; ++t) step(t);
    wait_vm<0>();   // no load may land in LDS after the workgroup ends
  }

  const int64_t coff = batch_off(z, a.inner_count, a.c_outer, a.c_inner, a.c_div);
#pragma clang loop unroll(full)
  for (int i = 0; i < IM; ++i)
#pragma clang loop unroll(full)
    for (int j = 0; j < JN; ++j)
      store_block<bf16_t>(a, acc[i][j], coff, m0 + wm * 128 + i * 32, n0 + wn * 128 + j * 32, lane);
}

template <bool AK, bool BKM>
void launch_w4k64_t(const GemmArgs& a, hipStream_t stream) {
  dim3 grid(ceil_div(a.N, 256), ceil_div(a.M, 256), a.nbatch);
  hipLaunchKernelGGL((gemm_bf16_w4k64<AK, BKM>), grid, dim3(256), 0, stream, a);
}
void launch_w4k64(const GemmArgs& a, hipStream_t stream) {
  const bool ak = a.A[0].s_k == 1, bk = a.B[0].s_k == 1;
  if (ak && bk) launch_w4k64_t<true, true>(a, stream);
  else if (ak && !bk) launch_w4k64_t<true, false>(a, stream);
  else if (!ak && bk) launch_w4k64_t<false, true>(a, stream);
  else launch_w4k64_t<false, false>(a, stream);
}

template <bool AK, bool BKM, int WN>
void launch_w4_t(const GemmArgs& a, hipStream_t stream) {
  dim3 grid(ceil_div(a.N, 256), ceil_div(a.M, 256), a.nbatch);
  hipLaunchKernelGGL((gemm_bf16_w4<AK, BKM, WN>), grid, dim3(128 * WN), 0, stream, a);
}
template <int WN>
void launch_w4(const GemmArgs& a, hipStream_t stream) {
  const bool ak = a.A[0].s_k == 1, bk = a.B[0].s_k == 1;
  if (ak && bk) launch_w4_t<true, true, WN>(a, stream);
  else if (ak && !bk) launch_w4_t<true, false, WN>(a, stream);
  else if (!ak && bk) launch_w4_t<false, true, WN>(a, stream);
  else launch_w4_t<false, false, WN>(a, stream);
}

template <int BN_, int WN>
void launch_dma(const GemmArgs& a, hipStream_t stream) {
  dim3 grid(ceil_div(a.N, BN_), ceil_div(a.M, 256), a.nbatch);
  dim3 block(64 * 2 * WN);
  const bool ak = a.A[0].s_k == 1, bk = a.B[0].s_k == 1;
  if (ak && bk) hipLaunchKernelGGL((gemm_bf16_dma<BN_, WN, true, true>), grid, block, 0, stream, a);
  else if (ak && !bk) hipLaunchKernelGGL((gemm_bf16_dma<BN_, WN, true, false>), grid, block, 0, stream, a);
  else if (!ak && bk) hipLaunchKernelGGL((gemm_bf16_dma<BN_, WN, false, true>), grid, block, 0, stream, a);
  else hipLaunchKernelGGL((gemm_bf16_dma<BN_, WN, false, false>), grid, block, 0, stream, a);
}

template <int BM_, int BN_, int WM, int WN>
void launch_big(const GemmArgs& a, hipStream_t stream) {
  dim3 grid(ceil_div(a.N, BN_), ceil_div(a.M, BM_), a.nbatch);
  dim3 block(64 * WM * WN);
  const bool ak = a.A[0].s_k == 1, bk = a.B[0].s_k == 1;
  if (ak && bk) hipLaunchKernelGGL((gemm_bf16_big<BM_, BN_, WM, WN, true, true>), grid, block, 0, stream, a);
  else if (ak && !bk) hipLaunchKernelGGL((gemm_bf16_big<BM_, BN_, WM, WN, true, false>), grid, block, 0, stream, a);
  else if (!ak && bk) hipLaunchKernelGGL((gemm_bf16_big<BM_, BN_, WM, WN, false, true>), grid, block, 0, stream, a);
  else hipLaunchKernelGGL((gemm_bf16_big<BM_, BN_, WM, WN, false, false>), grid, block, 0, stream, a);
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
  if (a.causal == CAUSAL_SKIP_UPPER && a.M > a.N) return "gemm: causal skip needs M <= N";
  if (a.tile < 0 || a.tile > 8) return "gemm: bad tile";
  if (a.tile >= 4 && (a.K % 32 || a.M < 8 || a.N < 8)) return "gemm: the DMA kernel needs K % 32 == 0";
  if (a.tile == 7 && a.K % 64) return "gemm: the 64-deep kernels need K % 64 == 0";
  if (a.tile == 7 && a.npairs == 2 &&
      (a.A[1].s_row != a.A[0].s_row || a.A[1].s_k != a.A[0].s_k || a.B[1].s_row != a.B[0].s_row ||
       a.B[1].s_k != a.B[0].s_k))
    return "gemm: the 64-deep kernels need equal operand strides in both pairs";
  return nullptr;
}

// The bf16 kernel a product runs on (the tile values of GemmArgs::tile).
static int bf16_tile(const GemmArgs& a) {
  int tile = a.tile;
  if (tile == 0 && a.M >= 256) {
    const int64_t t256 = (int64_t)ceil_div(a.M, 256) * ceil_div(a.N, 256) * a.nbatch;
    const int64_t t128 = (int64_t)ceil_div(a.M, 256) * ceil_div(a.N, 128) * a.nbatch;
    const bool dma = a.K % KT3 == 0;
    // 256 x 256 tiles once there are more than 128 of them; with fewer,
    // 256 x 128 tiles keep more of the 256 CUs busy.  Contractions up to
    // 4096 deep (the forward projections and the input gradients of
    // 2048-wide layers) run on eight wavefronts of 128 x 64, two per SIMD,
    // whose tiles spend less of their time in the prologue and the staged
    // epilogue; longer ones (the weight gradients, the input gradients of the
    // MLP and q/k/v) on four wavefronts of 128 x 128 (measured on the 1.3B
    // layer shapes, one and two operand pairs).
    if (a.N > 128 && t256 > 128) tile = dma ? (a.K <= 4096 ? 8 : 6) : 2;
    else if (t128 >= 64) tile = dma ? 5 : 3;
  }
  return tile;
}

template <typename T>
hipError_t gemm(const GemmArgs& a, hipStream_t stream) {
  if (a.M == 0 || a.N == 0) return hipSuccess;
  if constexpr (sizeof(T) == 2) {
    const int tile = bf16_tile(a);
    if (tile == 2) { launch_big<256, 256, 2, 4>(a, stream); return hipGetLastError(); }
    if (tile == 3) { launch_big<256, 128, 2, 2>(a, stream); return hipGetLastError(); }
    if (tile == 4) { launch_dma<256, 4>(a, stream); return hipGetLastError(); }
    if (tile == 5) { launch_dma<128, 2>(a, stream); return hipGetLastError(); }
    if (tile == 6) { launch_w4<2>(a, stream); return hipGetLastError(); }
    if (tile == 8) { launch_w4<4>(a, stream); return hipGetLastError(); }
    if (tile == 7) { launch_w4k64(a, stream); return hipGetLastError(); }
  }
  dim3 grid(ceil_div(a.N, BN), ceil_div(a.M, BM), a.nbatch);
  const bool ak = a.A[0].s_k == 1, bk = a.B[0].s_k == 1;
  if (ak && bk) hipLaunchKernelGGL((gemm_kernel<T, true, true>), grid, dim3(NT), 0, stream, a);
  else if (ak && !bk) hipLaunchKernelGGL((gemm_kernel<T, true, false>), grid, dim3(NT), 0, stream, a);
  else if (!ak && bk) hipLaunchKernelGGL((gemm_kernel<T, false, true>), grid, dim3(NT), 0, stream, a);
  else hipLaunchKernelGGL((gemm_kernel<T, false, false>), grid, dim3(NT), 0, stream, a);
  return hipGetLastError();
}

template <bool AK, bool BKM, int WN>
static void launch_w4_pair_t(const GemmArgs& a0, const GemmArgs& a1, int n0, int n1, hipStream_t stream) {
  hipLaunchKernelGGL((gemm_bf16_w4_pair<AK, BKM, WN>), dim3(n0 + n1), dim3(128 * WN), 0, stream, a0, a1, n0);
}
template <int WN>
static void launch_w4_pair(const GemmArgs& a0, const GemmArgs& a1, int n0, int n1, hipStream_t stream) {
  const bool ak = a0.A[0].s_k == 1, bk = a0.B[0].s_k == 1;
  if (ak && bk) launch_w4_pair_t<true, true, WN>(a0, a1, n0, n1, stream);
  else if (ak && !bk) launch_w4_pair_t<true, false, WN>(a0, a1, n0, n1, stream);
  else if (!ak && bk) launch_w4_pair_t<false, true, WN>(a0, a1, n0, n1, stream);
  else launch_w4_pair_t<false, false, WN>(a0, a1, n0, n1, stream);
}

template <typename T>
hipError_t gemm_pair(const GemmArgs& a0, const GemmArgs& a1, hipStream_t stream) {
  if constexpr (sizeof(T) == 2) {
    GemmArgs b = a1;
    b.tile = bf16_tile(a0);
    const bool one = (b.tile == 6 || b.tile == 8) && a0.M > 0 && a0.N > 0 && a1.M > 0 && a1.N > 0 &&
                     a0.causal == CAUSAL_NONE && a1.causal == CAUSAL_NONE &&
                     (a0.A[0].s_k == 1) == (a1.A[0].s_k == 1) && (a0.B[0].s_k == 1) == (a1.B[0].s_k == 1) &&
                     gemm_check<T>(b) == nullptr;
    if (one) {
      const int n0 = (int)(ceil_div(a0.M, 256) * ceil_div(a0.N, 256)) * a0.nbatch;
      const int n1 = (int)(ceil_div(a1.M, 256) * ceil_div(a1.N, 256)) * a1.nbatch;
      if (b.tile == 6) launch_w4_pair<2>(a0, b, n0, n1, stream);
      else launch_w4_pair<4>(a0, b, n0, n1, stream);
      return hipGetLastError();
    }
  }
  const hipError_t r = gemm<T>(a0, stream);
  return r != hipSuccess ? r : gemm<T>(a1, stream);
}

template hipError_t gemm<float>(const GemmArgs&, hipStream_t);
template hipError_t gemm<bf16_t>(const GemmArgs&, hipStream_t);
template hipError_t gemm_pair<float>(const GemmArgs&, const GemmArgs&, hipStream_t);
template hipError_t gemm_pair<bf16_t>(const GemmArgs&, const GemmArgs&, hipStream_t);
template const char* gemm_check<float>(const GemmArgs&);
template const char* gemm_check<bf16_t>(const GemmArgs&);

}  // namespace fdh
