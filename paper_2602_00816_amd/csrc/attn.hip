// Fused causal attention for the lockstep pair (bf16 operands, fp32
// accumulation): the forward output and the three input gradients without
// materialising the S x S score, probability or score-gradient matrices.
//
// The two gradient passes at theta +- eps v are carried as m = half sum and
// d = half difference of the two points' values (section 3.2, central
// difference of two backward passes).  With logits a = S.m * scale and
// b = S.d * scale of one query row, the two points' softmaxes are
// softmax(a + b) and softmax(a - b).  With Zc = sum e^a cosh b and
// Zs = sum e^a sinh b (row sums), D = Zc^2 - Zs^2, u = Zc / D, w = Zs / D:
//   P.m = e^a (u cosh b - w sinh b),   P.d = e^a (u sinh b - w cosh b)
// exactly, and with no difference of nearly equal numbers: the small
// quantities (b, sinh b, Zs) are carried directly.  The products follow the
// unfused path term by term (terms of order eps^2 relative are dropped):
//   O.m  = P.m V.m                 O.d  = P.m V.d + P.d V.m
//   dP.m = dO.m V.m^T              dP.d = dO.m V.d^T + dO.d V.m^T
//   dS.m = P.m (dP.m - D.m) + P.d (dP.d - D.d)
//   dS.d = P.m (dP.d - D.d) + P.d (dP.m - D.m)
//   with D.m = rowsum(dO.m O.m + dO.d O.d), D.d = rowsum(dO.m O.d + dO.d O.m)
//   dV.m = P.m^T dO.m              dV.d = P.m^T dO.d + P.d^T dO.m
//   dQ.m = dS.m K.m                dQ.d = dS.m K.d + dS.d K.m      (x scale)
//   dK.m = dS.m^T Q.m              dK.d = dS.m^T Q.d + dS.d^T Q.m  (x scale)
// The forward runs the softmax online over key blocks with two accumulators,
// Ac = sum e^a cosh b V.m and X = sum e^a (sinh b V.m + cosh b V.d), giving
// O.m = u Ac and O.d = u X - w Ac; the term -w sum e^a sinh b V.m of O.m is
// of order eps^2 relative, like the P.d V.d term the pair form drops.  The
// reference maximum of a moves lazily (see flash_fwd_kernel), and per query
// row (reference maximum, u, w) is stored for the backward.
//
// Three kernels, each with MFMA tiles oriented so that the probability-like
// accumulator feeds the next MFMA straight from registers: a 32x32 (16x16)
// accumulator holds, per lane, one column and 16 (4) rows; read in the order
// the accumulator holds them, its rows are a permutation of the next
// product's contraction index, and the other operand is read from LDS with
// the same permutation (transposing LDS reads, ds_read_b64_tr_b16).
//   flash_fwd   : one workgroup per 128 queries of one head, S^T = K Q^T tiles
//   flash_bwd_q : one workgroup per 128 queries, dQ^T = K^T dS^T
//   flash_bwd_kv: one workgroup per 64 keys of one key/value head (all query
//                 heads of its group), S = Q K^T tiles, dV = P^T dO, dK = dS^T Q
// K/V (or Q/dO) tiles are streamed into a double-buffered LDS ring by direct
// global-to-LDS loads.  LDS tiles are [rows][D] with the 16-byte chunk c of
// row r at c ^ f(r), f a bit reversal of low row bits (and, for the 16-row
// fragment reads of flash_bwd_kv, the variant described at tswz).
#include "common.h"
#include "kernels.h"

#include <type_traits>

namespace fdh {

namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef short v8i16 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16_t;
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr float NEG = -1.0e30f;   // masked logit (exp underflows to 0, no NaN)

// element offset of chunk `chunk` (8 elements) of row `row` in an LDS [rows][D] tile.
// SW = 0: chunk XOR the bit reversal of row & 15 (D = 128).  SW = 1 (the tiles
// read by 16x16 operands, D = 128): chunk XOR f(row & 7) with f's bits 3, 2 =
// bits 1, 0 of the row and bits 1, 0 both = bit 2.  Which lanes a 16-byte LDS
// read serves together is not documented; the bank-conflict counters show
// none for the 32-row reads (ld_k32, ld_t32) on SW = 0 and for the 16-row
// reads (ld_k16) and transposing reads (ld_t16) on SW = 1, and conflicts for
// 16-row reads on SW = 0 and for 16-byte reads of a layout with 64-byte rows.
// Every lane grouping that fits all of these (cosets of a subspace of the lane
// index bits, 64 or 32 banks) leaves the SW = 1 and SW = 2 16-row reads free.
// SW = 2 (the probability exchange tile of flash_bwd_kv8, D = 128): the f of
// SW = 1 with bit 1 flipped on rows 8..15 of every 16, so that sixteen
// consecutive rows take sixteen different chunk positions, which its 8-byte
// writes (lanes 16 g + i on row i) need.
template <int D, int SW = 0>
__device__ inline int tswz(int row, int chunk) {
  int f;
  if (D == 128 && SW >= 1) {
    const int r = row & 7;
    f = ((r & 3) << 2) | (((r >> 2) & 1) * 3);
    if (SW == 2) f ^= ((row >> 3) & 1) << 1;
  } else if (D == 128) {
    const int r = row & 15;
    f = ((r & 1) << 3) | ((r & 2) << 1) | ((r & 4) >> 1) | ((r & 8) >> 3);
  } else {
    const int r = (row >> 1) & 7;
    f = ((r & 1) << 2) | (r & 2) | ((r & 4) >> 2);
  }
  return row * D + ((chunk ^ f) << 3);
}

// 32x32x16 operand with the contraction along D: lane -> row r0 + lane % 32,
// columns 16 s + 8 (lane / 32) .. + 7
template <int D>
__device__ inline bf16x8_t ld_k32(const bf16_t* t, int r0, int s, int lane) {
  return *reinterpret_cast<const bf16x8_t*>(t + tswz<D>(r0 + (lane & 31), 2 * s + (lane >> 5)));
}
// 16x16x32 operand with the contraction along D: lane -> row r0 + lane % 16,
// columns 32 s + 8 (lane / 16) .. + 7
template <int D, int SW = 1>
__device__ inline bf16x8_t ld_k16(const bf16_t* t, int r0, int s, int lane) {
  return *reinterpret_cast<const bf16x8_t*>(t + tswz<D, SW>(r0 + (lane & 15), 4 * s + (lane >> 4)));
}
template <int D, int SW = 0>
__device__ inline v4i16 tr4(const bf16_t* t, int row, int col) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(t + tswz<D, SW>(row, col >> 3) + (col & 7)));
}
__device__ inline bf16x8_t cat(v4i16 a, v4i16 b) {
  const v8i16 v = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return __builtin_bit_cast(bf16x8_t, v);
}
// 32x32x16 operand with the contraction along the rows kk .. kk + 15 of the
// tile, in the row order of a 32x32 accumulator (lane half g: rows
// kk + 4 g .. + 3 and kk + 8 + 4 g .. + 3), column n0 + lane % 32
template <int D>
__device__ inline bf16x8_t ld_t32(const bf16_t* t, int kk, int n0, int lane) {
  const int g = lane >> 4, i = lane & 15;
  const int col = n0 + 16 * (g & 1) + 4 * (i & 3);
  const int lo = kk + 4 * (g >> 1) + (i >> 2);
  return cat(tr4<D>(t, lo, col), tr4<D>(t, lo + 8, col));
}
// 16x16x32 operand with the contraction along rows kk .. kk + 31 in the row
// order of two stacked 16x16 accumulators (lane quarter g: rows kk + 4 g .. + 3
// and kk + 16 + 4 g .. + 3), column n0 + lane % 16.  SWAP: quarters of odd
// parity (g = 1, 2) take the two row groups in the other order, matching an
// A operand whose 8-byte halves are exchanged on those quarters.
template <int D, bool SWAP = false>
__device__ inline bf16x8_t ld_t16(const bf16_t* t, int kk, int n0, int lane) {
  const int g = lane >> 4, i = lane & 15;
  const int col = n0 + 4 * (i & 3);
  const int sw = SWAP ? ((g ^ (g >> 1)) & 1) << 4 : 0;
  const int lo = kk + 4 * g + (i >> 2);
  return cat(tr4<D, 1>(t, lo + sw, col), tr4<D, 1>(t, lo + 16 - sw, col));
}

__device__ inline v4i16 pack4(const float* x) {
  v4i16 v;
#pragma unroll
  for (int j = 0; j < 4; ++j) v[j] = __builtin_bit_cast(short, (__bf16)x[j]);
  return v;
}
__device__ inline bf16x8_t pack8(const float* x) {
  bf16x8_t v;
#pragma unroll
  for (int j = 0; j < 8; ++j) v[j] = (__bf16)x[j];
  return v;
}

__device__ inline f32x16_t mma32(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ inline f32x4_t mma16(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// cosh and sinh of a logit difference b.  b is of order eps times a logit
// derivative; when every |b| of the wavefront is below SERIES_MAX the
// two-term series is exact to fp32 rounding (dropped terms b^4/120 and b^4/24
// relative, below 4e-8), otherwise the exponential form is used.
constexpr float SERIES_MAX = 1.f / 32.f;
template <bool SERIES>
__device__ inline void coshsinh(float b, float& c, float& s) {
  if constexpr (SERIES) {
    const float b2 = b * b;
    s = fmaf(b * b2, 1.f / 6.f, b);
    c = fmaf(b2, 0.5f, 1.f);
  } else {
    const float e = __expf(b), ie = __expf(-b);
    s = 0.5f * (e - ie);
    c = 0.5f * (e + ie);
  }
}

// Issue this wavefront's direct global-to-LDS loads of NTILE tiles of R rows
// x D bf16: tile i comes from rows src[i] + r * ld and lands swizzled at
// dst + i * R * D.  Each load moves 1 KB: 64 lanes x 16 bytes, lane l at
// +16 l in LDS, so each lane fetches the logical chunk that the swizzle puts
// at that position.  Completion is waited for with vmcnt before the barrier
// that publishes the tiles.
template <int D, int R, int NTILE, int SW = 0, int NWV = 4>
__device__ inline void dma_tiles(bf16_t* dst, const bf16_t* const (&src)[NTILE], int64_t ld, int wave, int lane) {
  constexpr int CPR = D / 8, RPI = 64 / CPR, IPT = R / RPI, NI = NTILE * IPT;
  static_assert(IPT % NWV == 0, "each tile's loads must split evenly over the wavefronts");
#pragma unroll
  for (int u = 0; u < NI / NWV; ++u) {
    const int tile = NWV * u / IPT;         // compile-time: wave < NWV never crosses a tile
    const int q = NWV * u % IPT + wave;
    const int row = q * RPI + lane / CPR, pch = lane % CPR;
    const int lch = (tswz<D, SW>(row, pch) - row * D) >> 3;   // the swizzle is an involution on chunks
    const bf16_t* g = src[tile] + (int64_t)row * ld + 8 * lch;
    const uint32_t la = (uint32_t)(uintptr_t)(lds_void_t*)(dst + tile * R * D + q * 512);
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off"
        :
        : "s"(__builtin_amdgcn_readfirstlane(la)), "v"(g)
        : "memory", "m0");
  }
}

// s_waitcnt with vmcnt = N (bits 3:0 and 15:14), expcnt and lgkmcnt at their maxima
template <int N>
__device__ inline void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Work item of a workgroup in a grid of nblk blocks (of queries or keys) x
// nhead heads, with the block index `blk` taken so that the longest items run
// first.  Workgroups are handed out in linear-id order and round-robin over
// the eight XCDs (id mod 8); ordering the items by block first gives every XCD
// the same mix of long and short items, where a (block fastest) ordering
// would give XCD k only the blocks congruent to k mod 8 and, under the causal
// mask, very different amounts of work.
__device__ inline void work_item(int nhead, int& blk, int& head) {
  const int id = blockIdx.x + gridDim.x * blockIdx.y;
  blk = id / nhead;
  head = id % nhead;
}

// ---------------------------------------------------------------------------
// forward
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void flash_fwd_kernel(FlashArgs a) {
  constexpr int KB = 32, KS = D / 16, NT = D / 32, TILE = KB * D;
  // K is one block ahead of V: iteration kb forms the scores of block kb + 1
  // while it turns the scores of block kb into the P V products.  Both rings
  // have R stages; the loads run R - 1 blocks ahead of their use.
  constexpr int R = 4;
  constexpr int LPP = D / 16;   // DMA instructions per wavefront per (K, V) block pair
  __shared__ __attribute__((aligned(1024))) bf16_t kring[R][2 * TILE];   // K.m K.d
  __shared__ __attribute__((aligned(1024))) bf16_t vring[R][2 * TILE];   // V.m V.d

  int qb, bh;
  work_item(gridDim.y, qb, bh);
  qb = gridDim.x - 1 - qb;   // longest rows first
  const int b = bh / a.Hq, h = bh % a.Hq, kh = h / a.G;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int q0 = qb * 128, qw = q0 + 32 * wave;
  const int64_t row0 = (int64_t)b * a.S;
  const int qi = qw + (lane & 31);

  // Q fragments (B operand of S^T = K Q^T), both points' halves
  bf16x8_t qm[KS], qd[KS];
  {
    const int64_t off = (row0 + qi) * a.ld + (int64_t)h * D + 8 * (lane >> 5);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      qm[s] = *reinterpret_cast<const bf16x8_t*>(a.qkv_m + off + 16 * s);
      qd[s] = *reinterpret_cast<const bf16x8_t*>(a.qkv_d + off + 16 * s);
      // keep the loop-invariant Q fragments in AGPRs (MFMA operands may come
      // from either file), leaving the VGPRs to the per-block values
      asm volatile("" : "+a"(qm[s]));
      asm volatile("" : "+a"(qd[s]));
    }
  }
  // Ac = sum e^a cosh b V.m;  X = sum e^a (sinh b V.m + cosh b V.d)
  f32x16_t Ac[NT], X[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) Ac[t][r] = X[t][r] = 0.f;
  float zc = 0.f, zs = 0.f;

  const int nkb = (q0 + 128) / KB;
  const int lastw = qw / KB;   // this wavefront's diagonal block
  constexpr float LOG2E = 1.4426950408889634f;
  // block j of K (or V) into stage j % R; past the last block the last block
  // is loaded again (never read), so every iteration issues the same number
  // of loads and the vmcnt waits are constants
  auto issue_k = [&](int j) {
    const int64_t r = row0 + (int64_t)min(j, nkb - 1) * KB;
    const bf16_t* src[2] = {a.qkv_m + r * a.ld + a.koff + kh * D, a.qkv_d + r * a.ld + a.koff + kh * D};
    dma_tiles<D, KB, 2>(kring[j % R], src, a.ld, wave, lane);
  };
  auto issue_v = [&](int j) {
    const int64_t r = row0 + (int64_t)min(j, nkb - 1) * KB;
    const bf16_t* src[2] = {a.qkv_m + r * a.ld + a.voff + kh * D, a.qkv_d + r * a.ld + a.voff + kh * D};
    dma_tiles<D, KB, 2>(vring[j % R], src, a.ld, wave, lane);
  };
  // raw scores of the block in kring[st]: sm = K.m q.m, sd = K.m q.d + K.d q.m
  auto scores = [&](int st, f32x16_t& sm, f32x16_t& sd) {
    const bf16_t* Km = kring[st];
    const bf16_t* Kd = Km + TILE;
#pragma unroll
    for (int r = 0; r < 16; ++r) sm[r] = sd[r] = 0.f;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const bf16x8_t km = ld_k32<D>(Km, 0, s, lane), kd = ld_k32<D>(Kd, 0, s, lane);
      sm = mma32(km, qm[s], sm);
      sd = mma32(km, qd[s], sd);
      sd = mma32(kd, qm[s], sd);
    }
  };

  // Reference maximum of the logits, moved lazily: only when a logit exceeds
  // it by more than 8 (e^8 ~ 3e3 keeps every term and row sum far from
  // overflow) are the accumulators and sums rescaled, which after the first
  // block is rare.  The accumulators live in VGPRs (this file is compiled with
  // VGPR-form MFMAs), so the rescale branch costs nothing when not taken.
  float mrun = NEG;
  f32x16_t sm, sd;
  // pair j = (K block j + 1, V block j); iteration kb issues pair kb + R - 1
  // and needs pair kb + 1 at its end
  issue_k(0);
#pragma unroll
  for (int j = 0; j < R - 1; ++j) {
    issue_k(j + 1);
    issue_v(j);
  }
  wait_vm<(R - 1) * LPP>();
  __syncthreads();
  scores(0, sm, sd);
  wait_vm<(R - 2) * LPP>();
  __syncthreads();
  for (int kb = 0; kb < nkb; ++kb) {
    issue_k(kb + R);
    issue_v(kb + R - 1);
    // every wavefront runs every block: past its diagonal all keys are masked
    // (exact zeros); a branch around the accumulator updates would make the
    // register allocator shuttle the accumulators through VGPRs each block
    if (kb >= lastw) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kb * KB + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        if (key > qi) sm[r] = NEG;
      }
    }
    float amax = NEG, bmax = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      amax = fmaxf(amax, sm[r]);
      bmax = fmaxf(bmax, fabsf(sd[r]));
    }
    amax *= a.scale;
    amax = fmaxf(amax, __shfl_xor(amax, 32, 64));
    if (__any(amax > mrun + 8.f)) {
      const float mnew = fmaxf(mrun, amax);
      const float alpha = __expf(mrun - mnew);
      mrun = mnew;
      zc *= alpha;
      zs *= alpha;
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          Ac[t][r] *= alpha;
          X[t][r] *= alpha;
        }
    }
    const float moff = -mrun * LOG2E;
    // The scores of the next block (the last iteration forms them from a
    // stale ring stage and drops them) overlap the element-wise terms of this
    // one, taken with the two-term series of cosh b and sinh b: per k step,
    // the fragment reads of the next step, the three score MFMAs and the terms
    // of 16 / KS elements, in this order (scheduling barriers keep the
    // compiler from regrouping them).
    f32x16_t smn, sdn;
#pragma unroll
    for (int r = 0; r < 16; ++r) smn[r] = sdn[r] = 0.f;
    float pc[16], ps[16];
    float zci = 0.f, zsi = 0.f;
    {
      constexpr int EPS = 16 / KS;   // elements per k step
      const bf16_t* Km = kring[(kb + 1) % R];
      const bf16_t* Kd = Km + TILE;
      bf16x8_t kmf[2], kdf[2];
      kmf[0] = ld_k32<D>(Km, 0, 0, lane);
      kdf[0] = ld_k32<D>(Kd, 0, 0, lane);
      auto term = [&](int r) {
        const float e = __builtin_amdgcn_exp2f(fmaf(sm[r], a.c_exp, moff));
        const float q2 = sd[r] * sd[r];
        pc[r] = e * fmaf(q2, a.c_cosh, 1.f);              // e^a cosh b
        ps[r] = e * (sd[r] * fmaf(q2, a.c_sinh, a.scale));  // e^a sinh b
        zci += pc[r];
        zsi += ps[r];
        // materialise the terms here: the fix-up branch below overwrites them,
        // and the compiler would otherwise sink this work past the MFMAs
        asm volatile("" : "+v"(pc[r]), "+v"(ps[r]), "+v"(zci), "+v"(zsi));
      };
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        if (s + 1 < KS) {
          kmf[(s + 1) & 1] = ld_k32<D>(Km, 0, s + 1, lane);
          kdf[(s + 1) & 1] = ld_k32<D>(Kd, 0, s + 1, lane);
        }
        smn = mma32(kmf[s & 1], qm[s], smn);
#pragma unroll
        for (int j = 0; j < EPS / 2; ++j) term(EPS * s + j);
        sdn = mma32(kmf[s & 1], qd[s], sdn);
#pragma unroll
        for (int j = EPS / 2; j < EPS; ++j) term(EPS * s + j);
        sdn = mma32(kdf[s & 1], qm[s], sdn);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    bf16x8_t bc[2], bs[2];
    bc[0] = pack8(pc); bc[1] = pack8(pc + 8);
    bs[0] = pack8(ps); bs[1] = pack8(ps + 8);
    // some |b| past the series range (never at the workloads' eps): redo the
    // terms with the exponential form
    if (__any(bmax * a.scale >= SERIES_MAX)) {
      zci = zsi = 0.f;
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2) {
        float pc[8], ps[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int r = 8 * t2 + j;
          const float e = __builtin_amdgcn_exp2f(fmaf(sm[r], a.c_exp, moff));
          float c, sn;
          coshsinh<false>(sd[r] * a.scale, c, sn);
          pc[j] = e * c;
          ps[j] = e * sn;
          zci += pc[j];
          zsi += ps[j];
        }
        bc[t2] = pack8(pc);
        bs[t2] = pack8(ps);
      }
    }
    zc += zci;
    zs += zsi;
    {
      const bf16_t* Vm = vring[kb % R];
      const bf16_t* Vd = Vm + TILE;
      bf16x8_t vmf[2], vdf[2];
      vmf[0] = ld_t32<D>(Vm, 0, 0, lane);
      vdf[0] = ld_t32<D>(Vd, 0, 0, lane);
#pragma unroll
      for (int i = 0; i < 2 * NT; ++i) {
        const int t2 = i / NT, t = i % NT;
        if (i + 1 < 2 * NT) {
          const int u2 = (i + 1) / NT, u = (i + 1) % NT;
          vmf[(i + 1) & 1] = ld_t32<D>(Vm, 16 * u2, 32 * u, lane);
          vdf[(i + 1) & 1] = ld_t32<D>(Vd, 16 * u2, 32 * u, lane);
        }
        Ac[t] = mma32(vmf[i & 1], bc[t2], Ac[t]);
        X[t] = mma32(vmf[i & 1], bs[t2], X[t]);
        X[t] = mma32(vdf[i & 1], bc[t2], X[t]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    sm = smn;
    sd = sdn;
    wait_vm<(R - 2) * LPP>();
    __syncthreads();
  }
  __builtin_amdgcn_s_waitcnt(0);   // the clamped reloads of the last iterations

  zc += __shfl_xor(zc, 32, 64);
  zs += __shfl_xor(zs, 32, 64);
  const float den = (zc - zs) * (zc + zs);
  const float u = zc / den, w = zs / den;
  const int64_t orow = (row0 + qi) * a.ldo + (int64_t)h * D + 4 * (lane >> 5);
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      uint16_t om[4], od[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 4 * g + e;
        om[e] = f32_to_bf16(u * Ac[t][r]);
        od[e] = f32_to_bf16(u * X[t][r] - w * Ac[t][r]);
      }
      const int64_t o = orow + 32 * t + 8 * g;
      *reinterpret_cast<uint2*>(a.o_m + o) = make_uint2(om[0] | ((uint32_t)om[1] << 16), om[2] | ((uint32_t)om[3] << 16));
      *reinterpret_cast<uint2*>(a.o_d + o) = make_uint2(od[0] | ((uint32_t)od[1] << 16), od[2] | ((uint32_t)od[3] << 16));
    }
  if (lane < 32) a.stats[(int64_t)bh * a.S + qi] = make_float4(mrun, u, w, 0.f);
}

// Forward with 16 queries per wavefront (D = 128): NW wavefronts, 16 NW
// queries of one head per workgroup, K and V blocks of 32 keys through a
// two-stage DMA ring.  Each wavefront forms S^T for the 32 keys and its 16
// queries (two 16-key halves); lane 16 g + i then holds keys 4g .. 4g + 3 and
// 16 + 4g .. + 3 of query i, which is the B operand of O^T = V^T P^T in the
// key order of the transposing V reads.  The output accumulators are O^T, so
// every lane holds its own query's columns (16 t + 4 g + r) and the lazy
// rescale by the running maximum stays lane-local; the maximum and the row
// sums are combined over the four lanes of a query with two shuffles.  Key
// blocks wholly above a wavefront's queries are skipped.  At under 256
// registers and 64 KB of LDS two workgroups share a CU.
template <int D, int NW>
__global__ __launch_bounds__(64 * NW, 2) void flash_fwd16_kernel(FlashArgs a) {
  static_assert(D == 128, "16-query forward is for head dimension 128");
  constexpr int KB = 32, KS = D / 32, TILE = KB * D, QS = 16 * NW, NT = D / 16;
  __shared__ __attribute__((aligned(1024))) bf16_t ring[2][4 * TILE];   // K.m K.d V.m V.d

  int qb, bh;
  work_item(gridDim.y, qb, bh);
  qb = gridDim.x - 1 - qb;   // longest rows first
  const int b = bh / a.Hq, h = bh % a.Hq, kh = h / a.G;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int q0 = qb * QS, qw = q0 + 16 * wave;
  const int64_t row0 = (int64_t)b * a.S;
  const int qi = qw + (lane & 15);

  bf16x8_t qm[KS], qd[KS];   // B operands of S^T = K Q^T
  {
    const int64_t off = (row0 + qi) * a.ld + (int64_t)h * D + 8 * (lane >> 4);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      qm[s] = *reinterpret_cast<const bf16x8_t*>(a.qkv_m + off + 32 * s);
      qd[s] = *reinterpret_cast<const bf16x8_t*>(a.qkv_d + off + 32 * s);
    }
  }
  // Ac = sum e^a cosh b V.m;  X = sum e^a (sinh b V.m + cosh b V.d), as O^T
  f32x4_t Ac[NT], X[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) Ac[t][r] = X[t][r] = 0.f;
  float zc = 0.f, zs = 0.f;
  constexpr float LOG2E = 1.4426950408889634f;
  float mrun = NEG;   // reference maximum of the scaled logits, moved lazily (see flash_fwd_kernel)

  const int nkb = (q0 + QS) / KB;
  const int lastw = (qw + 15) / KB;   // this wavefront's last key block
  auto issue = [&](int kb) {
    const int64_t r = row0 + (int64_t)kb * KB;
    const bf16_t* src[4] = {a.qkv_m + r * a.ld + a.koff + kh * D, a.qkv_d + r * a.ld + a.koff + kh * D,
                            a.qkv_m + r * a.ld + a.voff + kh * D, a.qkv_d + r * a.ld + a.voff + kh * D};
    dma_tiles<D, KB, 4, 1, NW>(ring[kb & 1], src, a.ld, wave, lane);
  };
  issue(0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int kb = 0; kb < nkb; ++kb) {
    if (kb + 1 < nkb) issue(kb + 1);
    if (kb <= lastw) {
      const bf16_t* Km = ring[kb & 1];
      const bf16_t* Kd = Km + TILE;
      const bf16_t* Vm = Km + 2 * TILE;
      const bf16_t* Vd = Km + 3 * TILE;
      f32x4_t sm[2], sd[2];   // raw scores: sm = K.m q.m, sd = K.m q.d + K.d q.m
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
#pragma unroll
        for (int r = 0; r < 4; ++r) sm[hf][r] = sd[hf][r] = 0.f;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const bf16x8_t km = ld_k16<D>(Km, 16 * hf, s, lane), kd = ld_k16<D>(Kd, 16 * hf, s, lane);
          sm[hf] = mma16(km, qm[s], sm[hf]);
          sd[hf] = mma16(km, qd[s], sd[hf]);
          sd[hf] = mma16(kd, qm[s], sd[hf]);
        }
        if (kb * KB + 16 * hf + 15 > qw) {
          const int key0 = kb * KB + 16 * hf + 4 * (lane >> 4);
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (key0 + r > qi) sm[hf][r] = NEG;
        }
      }
      float amax = NEG, bmax = 0.f;
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          amax = fmaxf(amax, sm[hf][r]);
          bmax = fmaxf(bmax, fabsf(sd[hf][r]));
        }
      amax *= a.scale;
      amax = fmaxf(amax, __shfl_xor(amax, 16, 64));
      amax = fmaxf(amax, __shfl_xor(amax, 32, 64));
      if (__any(amax > mrun + 8.f)) {
        const float mnew = fmaxf(mrun, amax);
        const float alpha = __expf(mrun - mnew);
        mrun = mnew;
        zc *= alpha;
        zs *= alpha;
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            Ac[t][r] *= alpha;
            X[t][r] *= alpha;
          }
      }
      const float moff = -mrun * LOG2E;
      float pc[2][4], ps[2][4];
      if (!__any(bmax * a.scale >= SERIES_MAX)) {
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float e = __builtin_amdgcn_exp2f(fmaf(sm[hf][r], a.c_exp, moff));
            const float q2 = sd[hf][r] * sd[hf][r];
            pc[hf][r] = e * fmaf(q2, a.c_cosh, 1.f);                  // e^a cosh b
            ps[hf][r] = e * (sd[hf][r] * fmaf(q2, a.c_sinh, a.scale));  // e^a sinh b
          }
      } else {
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float e = __builtin_amdgcn_exp2f(fmaf(sm[hf][r], a.c_exp, moff));
            float c, sn;
            coshsinh<false>(sd[hf][r] * a.scale, c, sn);
            pc[hf][r] = e * c;
            ps[hf][r] = e * sn;
          }
      }
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          zc += pc[hf][r];
          zs += ps[hf][r];
        }
      const bf16x8_t bc = cat(pack4(pc[0]), pack4(pc[1])), bs = cat(pack4(ps[0]), pack4(ps[1]));
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const bf16x8_t vmt = ld_t16<D>(Vm, 0, 16 * t, lane), vdt = ld_t16<D>(Vd, 0, 16 * t, lane);
        Ac[t] = mma16(vmt, bc, Ac[t]);
        X[t] = mma16(vmt, bs, X[t]);
        X[t] = mma16(vdt, bc, X[t]);
      }
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();   // the ring stage is free again
  }

  zc += __shfl_xor(zc, 16, 64);
  zs += __shfl_xor(zs, 16, 64);
  zc += __shfl_xor(zc, 32, 64);
  zs += __shfl_xor(zs, 32, 64);
  const float den = (zc - zs) * (zc + zs);
  const float u = zc / den, w = zs / den;
  const int64_t orow = (row0 + qi) * a.ldo + (int64_t)h * D + 4 * (lane >> 4);
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    uint16_t om[4], od[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      om[r] = f32_to_bf16(u * Ac[t][r]);
      od[r] = f32_to_bf16(u * X[t][r] - w * Ac[t][r]);
    }
    const int64_t o = orow + 16 * t;
    *reinterpret_cast<uint2*>(a.o_m + o) = make_uint2(om[0] | ((uint32_t)om[1] << 16), om[2] | ((uint32_t)om[3] << 16));
    *reinterpret_cast<uint2*>(a.o_d + o) = make_uint2(od[0] | ((uint32_t)od[1] << 16), od[2] | ((uint32_t)od[3] << 16));
  }
  if (lane < 16) a.stats[(int64_t)bh * a.S + qi] = make_float4(mrun, u, w, 0.f);
}

// ---------------------------------------------------------------------------
// backward: row terms D.m, D.d
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void flash_delta_kernel(FlashArgs a, int nrows) {
  // 16 lanes per (token, head) row; D / 16 elements per lane
  constexpr int E = D / 16;
  const int64_t row = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
  if (row >= nrows) return;
  const int sub = threadIdx.x & 15;
  const int64_t t = row / a.Hq;
  const int h = (int)(row % a.Hq);
  const int64_t off = t * a.ldo + (int64_t)h * D + sub * E;
  float dm = 0.f, dd = 0.f;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const float om = bf16_to_f32(a.o_m[off + e]), od = bf16_to_f32(a.o_d[off + e]);
    const float gm = bf16_to_f32(a.do_m[off + e]), gd = bf16_to_f32(a.do_d[off + e]);
    dm += gm * om + gd * od;
    dd += gm * od + gd * om;
  }
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) {
    dm += __shfl_xor(dm, o, 64);
    dd += __shfl_xor(dd, o, 64);
  }
  if (sub == 0) {
    const int b = (int)(t / a.S), i = (int)(t % a.S);
    a.delta[((int64_t)b * a.Hq + h) * a.S + i] = make_float2(dm, dd);
  }
}

// ---------------------------------------------------------------------------
// backward: dQ
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void flash_bwd_q_kernel(FlashArgs a) {
  constexpr int KB = 32, KS = D / 16, NT = D / 32, TILE = KB * D;
  __shared__ __attribute__((aligned(1024))) bf16_t ring[2][4 * TILE];   // K.m K.d V.m V.d

  int qb, bh;
  work_item(gridDim.y, qb, bh);
  qb = gridDim.x - 1 - qb;   // longest rows first
  const int b = bh / a.Hq, h = bh % a.Hq, kh = h / a.G;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int q0 = qb * 128, qw = q0 + 32 * wave;
  const int64_t row0 = (int64_t)b * a.S;
  const int qi = qw + (lane & 31);

  bf16x8_t qm[KS], qd[KS], gm[KS], gd[KS];   // Q and dO fragments (B operands)
  {
    const int64_t off = (row0 + qi) * a.ld + (int64_t)h * D + 8 * (lane >> 5);
    const int64_t offo = (row0 + qi) * a.ldo + (int64_t)h * D + 8 * (lane >> 5);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      qm[s] = *reinterpret_cast<const bf16x8_t*>(a.qkv_m + off + 16 * s);
      qd[s] = *reinterpret_cast<const bf16x8_t*>(a.qkv_d + off + 16 * s);
      gm[s] = *reinterpret_cast<const bf16x8_t*>(a.do_m + offo + 16 * s);
      gd[s] = *reinterpret_cast<const bf16x8_t*>(a.do_d + offo + 16 * s);
    }
  }
  const float4 st = a.stats[(int64_t)bh * a.S + qi];
  const float2 dl = a.delta[(int64_t)bh * a.S + qi];
  f32x16_t Qm[NT], Qd[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) Qm[t][r] = Qd[t][r] = 0.f;

  const int nkb = (q0 + 128) / KB;
  const int lastw = qw / KB;
  auto issue = [&](int kb) {
    const int64_t r = row0 + (int64_t)kb * KB;
    const bf16_t* src[4] = {a.qkv_m + r * a.ld + a.koff + kh * D, a.qkv_d + r * a.ld + a.koff + kh * D,
                            a.qkv_m + r * a.ld + a.voff + kh * D, a.qkv_d + r * a.ld + a.voff + kh * D};
    dma_tiles<D, KB, 4>(ring[kb & 1], src, a.ld, wave, lane);
  };
  issue(0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int kb = 0; kb < nkb; ++kb) {
    if (kb + 1 < nkb) issue(kb + 1);
    {   // every block, masked past the diagonal (see the forward kernel)
      const bf16_t* Km = ring[kb & 1];
      const bf16_t* Kd = Km + TILE;
      const bf16_t* Vm = Km + 2 * TILE;
      const bf16_t* Vd = Km + 3 * TILE;
      f32x16_t sm, sd, pm, pd;
#pragma unroll
      for (int r = 0; r < 16; ++r) sm[r] = sd[r] = pm[r] = pd[r] = 0.f;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const bf16x8_t km = ld_k32<D>(Km, 0, s, lane), kd = ld_k32<D>(Kd, 0, s, lane);
        sm = mma32(km, qm[s], sm);
        sd = mma32(km, qd[s], sd);
        sd = mma32(kd, qm[s], sd);
        const bf16x8_t vm = ld_k32<D>(Vm, 0, s, lane), vd = ld_k32<D>(Vd, 0, s, lane);
        pm = mma32(vm, gm[s], pm);
        pd = mma32(vm, gd[s], pd);
        pd = mma32(vd, gm[s], pd);
      }
      const bool diag = kb >= lastw;
      float bmax = 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        sm[r] *= a.scale;
        sd[r] *= a.scale;
        bmax = fmaxf(bmax, fabsf(sd[r]));
      }
      if (diag) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kb * KB + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
          if (key > qi) sm[r] = NEG;
        }
      }
      float gsm[16], gsd[16];
      auto terms = [&](auto ser) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float e = __expf(sm[r] - st.x);
          float c, sn;
          coshsinh<decltype(ser)::value>(sd[r], c, sn);
          const float Pm = e * (c * st.y - sn * st.z), Pd = e * (sn * st.y - c * st.z);
          const float xm = pm[r] - dl.x, xd = pd[r] - dl.y;
          gsm[r] = Pm * xm + Pd * xd;
          gsd[r] = Pm * xd + Pd * xm;
        }
      };
      if (!__any(bmax >= SERIES_MAX)) terms(std::true_type{});
      else terms(std::false_type{});
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2) {
        const bf16x8_t bm = pack8(gsm + 8 * t2), bd = pack8(gsd + 8 * t2);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const bf16x8_t km = ld_t32<D>(Km, 16 * t2, 32 * t, lane), kd = ld_t32<D>(Kd, 16 * t2, 32 * t, lane);
          Qm[t] = mma32(km, bm, Qm[t]);
          Qd[t] = mma32(kd, bm, Qd[t]);
          Qd[t] = mma32(km, bd, Qd[t]);
        }
      }
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }

  const int64_t grow = (row0 + qi) * a.ldg + (int64_t)h * D + 4 * (lane >> 5);
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int64_t o = grow + 32 * t + 8 * g;
      *reinterpret_cast<float4*>(a.g_m + o) =
          make_float4(Qm[t][4 * g] * a.scale, Qm[t][4 * g + 1] * a.scale, Qm[t][4 * g + 2] * a.scale,
                      Qm[t][4 * g + 3] * a.scale);
      *reinterpret_cast<float4*>(a.g_d + o) =
          make_float4(Qd[t][4 * g] * a.scale, Qd[t][4 * g + 1] * a.scale, Qd[t][4 * g + 2] * a.scale,
                      Qd[t][4 * g + 3] * a.scale);
    }
}

// dQ with 16 queries per wavefront (D = 128): NW wavefronts, 16 NW queries of
// one head per workgroup, key blocks of 32 through the DMA ring.  Each
// wavefront forms S^T and dP^T for the 32 keys of the block and its 16
// queries (two 16-key halves, query and output-gradient fragments in
// registers), and the score gradients of the two halves, rounded to bf16,
// are already the A operand of dQ = dS K in the key order of the transposing
// reads: lane 16 g + i holds keys 4g .. 4g + 3 and 16 + 4g .. + 3 of query i.
// So no exchange through LDS and one barrier per block.  Key blocks wholly
// above a wavefront's queries are skipped.  About 220 registers: with four
// wavefronts, two workgroups share a CU and their barriers are independent.
template <int D, int NW>
__global__ __launch_bounds__(64 * NW, 2) void flash_bwd_q16_kernel(FlashArgs a) {
  static_assert(D == 128, "16-query dQ is for head dimension 128");
  constexpr int KB = 32, KS = D / 32, TILE = KB * D, QS = 16 * NW, NT = D / 16;
  __shared__ __attribute__((aligned(1024))) bf16_t ring[2][4 * TILE];   // K.m K.d V.m V.d

  int qb, bh;
  work_item(gridDim.y, qb, bh);
  qb = gridDim.x - 1 - qb;   // longest rows first
  const int b = bh / a.Hq, h = bh % a.Hq, kh = h / a.G;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int q0 = qb * QS, qw = q0 + 16 * wave;
  const int64_t row0 = (int64_t)b * a.S;
  const int qi = qw + (lane & 15);

  bf16x8_t qm[KS], qd[KS], gm[KS], gd[KS];   // B operands of S^T = K Q^T, dP^T = V dO^T
  {
    const int64_t off = (row0 + qi) * a.ld + (int64_t)h * D + 8 * (lane >> 4);
    const int64_t offo = (row0 + qi) * a.ldo + (int64_t)h * D + 8 * (lane >> 4);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      qm[s] = *reinterpret_cast<const bf16x8_t*>(a.qkv_m + off + 32 * s);
      qd[s] = *reinterpret_cast<const bf16x8_t*>(a.qkv_d + off + 32 * s);
      gm[s] = *reinterpret_cast<const bf16x8_t*>(a.do_m + offo + 32 * s);
      gd[s] = *reinterpret_cast<const bf16x8_t*>(a.do_d + offo + 32 * s);
    }
  }
  const float4 st = a.stats[(int64_t)bh * a.S + qi];
  const float2 dl = a.delta[(int64_t)bh * a.S + qi];
  // accumulators t: queries qw + 4 (lane / 16) + r, columns 16 t + lane % 16
  f32x4_t Qm[NT], Qd[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) Qm[t][r] = Qd[t][r] = 0.f;

  const int nkb = (q0 + QS) / KB;
  const int lastw = (qw + 15) / KB;   // this wavefront's last key block
  auto issue = [&](int kb) {
    const int64_t r = row0 + (int64_t)kb * KB;
    const bf16_t* src[4] = {a.qkv_m + r * a.ld + a.koff + kh * D, a.qkv_d + r * a.ld + a.koff + kh * D,
                            a.qkv_m + r * a.ld + a.voff + kh * D, a.qkv_d + r * a.ld + a.voff + kh * D};
    dma_tiles<D, KB, 4, 1, NW>(ring[kb & 1], src, a.ld, wave, lane);
  };
  issue(0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int kb = 0; kb < nkb; ++kb) {
    if (kb + 1 < nkb) issue(kb + 1);
    if (kb <= lastw) {
      const bf16_t* Km = ring[kb & 1];
      const bf16_t* Kd = Km + TILE;
      const bf16_t* Vm = Km + 2 * TILE;
      const bf16_t* Vd = Km + 3 * TILE;
      float gsm[2][4], gsd[2][4];
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {   // keys kb * 32 + 16 hf .. + 15
        f32x4_t sm, sd, pm, pd;
#pragma unroll
        for (int r = 0; r < 4; ++r) sm[r] = sd[r] = pm[r] = pd[r] = 0.f;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const bf16x8_t km = ld_k16<D>(Km, 16 * hf, s, lane), kd = ld_k16<D>(Kd, 16 * hf, s, lane);
          sm = mma16(km, qm[s], sm);
          sd = mma16(km, qd[s], sd);
          sd = mma16(kd, qm[s], sd);
          const bf16x8_t vm = ld_k16<D>(Vm, 16 * hf, s, lane), vd = ld_k16<D>(Vd, 16 * hf, s, lane);
          pm = mma16(vm, gm[s], pm);
          pd = mma16(vm, gd[s], pd);
          pd = mma16(vd, gm[s], pd);
        }
        float bmax = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          sm[r] *= a.scale;
          sd[r] *= a.scale;
          bmax = fmaxf(bmax, fabsf(sd[r]));
        }
        const int key0 = kb * KB + 16 * hf + 4 * (lane >> 4);   // keys of this lane's rows: key0 + r
        if (kb * KB + 16 * hf + 15 > qw) {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (key0 + r > qi) sm[r] = NEG;
        }
        auto terms = [&](auto ser) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float e = __expf(sm[r] - st.x);
            float c, sn;
            coshsinh<decltype(ser)::value>(sd[r], c, sn);
            const float Pm = e * (c * st.y - sn * st.z), Pd = e * (sn * st.y - c * st.z);
            const float xm = pm[r] - dl.x, xd = pd[r] - dl.y;
            gsm[hf][r] = Pm * xm + Pd * xd;
            gsd[hf][r] = Pm * xd + Pd * xm;
          }
        };
        if (!__any(bmax >= SERIES_MAX)) terms(std::true_type{});
        else terms(std::false_type{});
      }
      const bf16x8_t dsm = cat(pack4(gsm[0]), pack4(gsm[1])), dsd = cat(pack4(gsd[0]), pack4(gsd[1]));
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const bf16x8_t kmt = ld_t16<D>(Km, 0, 16 * t, lane), kdt = ld_t16<D>(Kd, 0, 16 * t, lane);
        Qm[t] = mma16(dsm, kmt, Qm[t]);
        Qd[t] = mma16(dsm, kdt, Qd[t]);
        Qd[t] = mma16(dsd, kmt, Qd[t]);
      }
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();   // the ring stage is free again
  }

#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t o = (row0 + qw + 4 * (lane >> 4) + r) * a.ldg + (int64_t)h * D + 16 * t + (lane & 15);
      a.g_m[o] = Qm[t][r] * a.scale;
      a.g_d[o] = Qd[t][r] * a.scale;
    }
}

// ---------------------------------------------------------------------------
// backward: dK, dV (summed over the query heads that share the key/value head)
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void flash_bwd_kv_kernel(FlashArgs a) {
  constexpr int QB = 32, KS = D / 32, NT = D / 16, TILE = QB * D;
  __shared__ __attribute__((aligned(1024))) bf16_t ring[2][4 * TILE];   // Q.m Q.d dO.m dO.d
  __shared__ float4 sst[2][QB];                                         // m, u, w, D.m
  __shared__ __attribute__((aligned(16))) float sdd[2][QB];             // D.d

  int kblk, bkh;
  work_item(gridDim.y, kblk, bkh);   // lowest keys (most queries) first
  const int b = bkh / a.Hk, kh = bkh % a.Hk;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int k0 = kblk * 64, kw = k0 + 16 * wave;
  const int64_t row0 = (int64_t)b * a.S;
  const int kj = kw + (lane & 15);

  // K and V fragments of this wavefront's 16 keys (B operands of S = Q K^T, dP = dO V^T)
  bf16x8_t km[KS], kd[KS], vm[KS], vd[KS];
  {
    const int64_t r = (row0 + kj) * a.ld + kh * D + 8 * (lane >> 4);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      km[s] = *reinterpret_cast<const bf16x8_t*>(a.qkv_m + r + a.koff + 32 * s);
      kd[s] = *reinterpret_cast<const bf16x8_t*>(a.qkv_d + r + a.koff + 32 * s);
      vm[s] = *reinterpret_cast<const bf16x8_t*>(a.qkv_m + r + a.voff + 32 * s);
      vd[s] = *reinterpret_cast<const bf16x8_t*>(a.qkv_d + r + a.voff + 32 * s);
    }
  }
  f32x4_t Vm_[NT], Vd_[NT], Km_[NT], Kd_[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) Vm_[t][r] = Vd_[t][r] = Km_[t][r] = Kd_[t][r] = 0.f;

  const int nqb = (a.S - k0) / QB;   // query blocks from the first key on, per head
  const int total = nqb * a.G;
  auto issue = [&](int it) {
    const int g = it / nqb, qbk = it % nqb;
    const int h = kh * a.G + g, q0 = k0 + qbk * QB;
    const int64_t r = row0 + q0;
    const bf16_t* src[4] = {a.qkv_m + r * a.ld + (int64_t)h * D, a.qkv_d + r * a.ld + (int64_t)h * D,
                            a.do_m + r * a.ldo + (int64_t)h * D, a.do_d + r * a.ldo + (int64_t)h * D};
    // the two row strides differ: issue the Q and dO pairs separately
    const bf16_t* sq[2] = {src[0], src[1]};
    const bf16_t* so[2] = {src[2], src[3]};
    dma_tiles<D, QB, 2, 1>(ring[it & 1], sq, a.ld, wave, lane);
    dma_tiles<D, QB, 2, 1>(ring[it & 1] + 2 * TILE, so, a.ldo, wave, lane);
  };
  // row terms of the next block: loaded into registers with its tiles, written
  // to LDS after this block's compute (the load's wait would otherwise also
  // wait for the tile loads issued just before it)
  float4 nst = make_float4(0.f, 0.f, 0.f, 0.f);
  float ndd = 0.f;
  auto load_rows = [&](int it) {
    if (tid < QB) {
      const int g = it / nqb, qbk = it % nqb;
      const int64_t si = ((int64_t)b * a.Hq + kh * a.G + g) * a.S + k0 + qbk * QB + tid;
      const float4 st = a.stats[si];
      const float2 dl = a.delta[si];
      nst = make_float4(st.x, st.y, st.z, dl.x);
      ndd = dl.y;
    }
  };
  auto store_rows = [&](int it) {
    if (tid < QB) {
      sst[it & 1][tid] = nst;
      sdd[it & 1][tid] = ndd;
    }
  };
  load_rows(0);
  issue(0);
  __builtin_amdgcn_s_waitcnt(0);
  store_rows(0);
  __syncthreads();
  for (int it = 0; it < total; ++it) {
    if (it + 1 < total) {
      load_rows(it + 1);
      issue(it + 1);
    }
    const int q0 = k0 + (it % nqb) * QB;
    {   // every block; blocks wholly before this wavefront's keys are fully masked
      const bf16_t* Qm = ring[it & 1];
      const bf16_t* Qd = Qm + TILE;
      const bf16_t* Om = Qm + 2 * TILE;
      const bf16_t* Od = Qm + 3 * TILE;
      f32x4_t sm[2], sd[2], pm[2], pd[2];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
#pragma unroll
        for (int r = 0; r < 4; ++r) sm[qt][r] = sd[qt][r] = pm[qt][r] = pd[qt][r] = 0.f;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const bf16x8_t qa = ld_k16<D>(Qm, 16 * qt, s, lane), qb_ = ld_k16<D>(Qd, 16 * qt, s, lane);
          sm[qt] = mma16(qa, km[s], sm[qt]);
          sd[qt] = mma16(qa, kd[s], sd[qt]);
          sd[qt] = mma16(qb_, km[s], sd[qt]);
          const bf16x8_t oa = ld_k16<D>(Om, 16 * qt, s, lane), ob = ld_k16<D>(Od, 16 * qt, s, lane);
          pm[qt] = mma16(oa, vm[s], pm[qt]);
          pd[qt] = mma16(oa, vd[s], pd[qt]);
          pd[qt] = mma16(ob, vm[s], pd[qt]);
        }
      }
      const bool diag = q0 < kw + 16;
      float bmax = 0.f;
#pragma unroll
      for (int qt = 0; qt < 2; ++qt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          sm[qt][r] *= a.scale;
          sd[qt][r] *= a.scale;
          bmax = fmaxf(bmax, fabsf(sd[qt][r]));
        }
      if (diag) {
#pragma unroll
        for (int qt = 0; qt < 2; ++qt)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (q0 + 16 * qt + 4 * (lane >> 4) + r < kj) sm[qt][r] = NEG;
      }
      float Pm[8], Pd[8], gsm[8], gsd[8];   // rows in accumulator order: (qt, r) -> 4 qt + r
      auto terms = [&](auto ser) {
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
          const float4 ddv = *reinterpret_cast<const float4*>(&sdd[it & 1][16 * qt + 4 * (lane >> 4)]);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float4 st = sst[it & 1][16 * qt + 4 * (lane >> 4) + r];
            const float dd = r == 0 ? ddv.x : (r == 1 ? ddv.y : (r == 2 ? ddv.z : ddv.w));
            const float e = __expf(sm[qt][r] - st.x);
            float c, sn;
            coshsinh<decltype(ser)::value>(sd[qt][r], c, sn);
            const float P_m = e * (c * st.y - sn * st.z), P_d = e * (sn * st.y - c * st.z);
            const float xm = pm[qt][r] - st.w, xd = pd[qt][r] - dd;
            Pm[4 * qt + r] = P_m;
            Pd[4 * qt + r] = P_d;
            gsm[4 * qt + r] = P_m * xm + P_d * xd;
            gsd[4 * qt + r] = P_m * xd + P_d * xm;
          }
        }
      };
      if (!__any(bmax >= SERIES_MAX)) terms(std::true_type{});
      else terms(std::false_type{});
      const bf16x8_t apm = pack8(Pm), apd = pack8(Pd), asm_ = pack8(gsm), asd = pack8(gsd);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const bf16x8_t om = ld_t16<D>(Om, 0, 16 * t, lane), od = ld_t16<D>(Od, 0, 16 * t, lane);
        Vm_[t] = mma16(apm, om, Vm_[t]);
        Vd_[t] = mma16(apm, od, Vd_[t]);
        Vd_[t] = mma16(apd, om, Vd_[t]);
        const bf16x8_t qa = ld_t16<D>(Qm, 0, 16 * t, lane), qb_ = ld_t16<D>(Qd, 0, 16 * t, lane);
        Km_[t] = mma16(asm_, qa, Km_[t]);
        Kd_[t] = mma16(asm_, qb_, Kd_[t]);
        Kd_[t] = mma16(asd, qa, Kd_[t]);
      }
    }
    __builtin_amdgcn_s_waitcnt(0);
    if (it + 1 < total) store_rows(it + 1);
    __syncthreads();
  }

  // accumulator (t, r): key kw + 4 (lane / 16) + r, column 16 t + lane % 16
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t o = (row0 + kw + 4 * (lane >> 4) + r) * a.ldg + kh * D + 16 * t + (lane & 15);
      a.g_m[o + a.koff] = Km_[t][r] * a.scale;
      a.g_d[o + a.koff] = Kd_[t][r] * a.scale;
      a.g_m[o + a.voff] = Vm_[t][r];
      a.g_d[o + a.voff] = Vd_[t][r];
    }
}

// dK/dV with the probabilities shared through LDS (D = 128): 64 keys of one
// key/value head per workgroup of eight wavefronts, two per SIMD (about 220
// registers each), where the one-workgroup-of-four form runs one wavefront
// per SIMD and hides nothing.  Score phase: wavefront w forms S, dP, P and dS
// for 16 keys (group w / 2) and 16 of the 32 queries of the block (half
// w % 2), as flash_bwd_kv_kernel does for both halves; it writes its P.m, P.d,
// dS.m, dS.d fragments (8 bytes per lane, in the query order of the
// transposing reads) to an LDS buffer of the workgroup.  After a barrier
// wavefront w accumulates dV and dK for all 64 keys on 16 of the 128 columns
// (16 w .. 16 w + 15): its transposing reads of the Q and dO tiles cover an
// eighth of them, and the P/dS operands come back as 16-byte reads.
// One barrier per query block: the Q/dO tiles go through a three-stage ring
// (the block after the next is loaded only once every wavefront has passed
// the barrier that follows its last reads of that stage) and the P buffer is
// doubled, so a wavefront may start the score phase of the next block while
// others still accumulate this one; each wavefront waits for its own loads of
// the next block before the barrier, which then publishes them.  With a
// second barrier at the end of every block (two stages, one buffer) the
// kernel took 5% longer.
// P buffer (each of the two): one [64 keys][128] bf16 tile with the SW = 2 swizzle, operand o
// (P.m, P.d, dS.m, dS.d) in chunks 4o .. 4o + 3, chunk 4o + g of key row r
// holding queries 4g .. 4g + 3 and 16 + 4g .. + 3, in that order when g has
// even parity and swapped when odd (the B operands are read with the same
// swap); the accumulation phase reads it with ld_k16.  A wavefront of the
// score phase fills one 8-byte half of each chunk it touches: with the half
// fixed per wavefront the writes of 32 lanes met only half of the banks, and
// a quarter of the LDS cycles went to bank conflicts.

template <int D>
__global__ __launch_bounds__(512, 1) void flash_bwd_kv8_kernel(FlashArgs a) {
  static_assert(D == 128, "eight-wavefront dK/dV is for head dimension 128");
  constexpr int QB = 32, KS = D / 32, TILE = QB * D, KEYS = 64;
  __shared__ __attribute__((aligned(1024))) bf16_t ring[3][4 * TILE];     // Q.m Q.d dO.m dO.d
  __shared__ __attribute__((aligned(1024))) bf16_t pbufs[2][KEYS * D];    // P.m P.d dS.m dS.d
  __shared__ float4 sst[2][QB];                                           // m, u, w, D.m
  __shared__ __attribute__((aligned(16))) float sdd[2][QB];               // D.d

  int kblk, bkh;
  work_item(gridDim.y, kblk, bkh);   // lowest keys (most queries) first
  const int b = bkh / a.Hk, kh = bkh % a.Hk;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kg = wave >> 1, qt = wave & 1;   // score phase: key group and query half
  const int k0 = kblk * KEYS, kw = k0 + 16 * kg;
  const int64_t row0 = (int64_t)b * a.S;
  const int kj = kw + (lane & 15);

  // K and V fragments of this wavefront's 16 keys (B operands of S = Q K^T, dP = dO V^T)
  bf16x8_t km[KS], kd[KS], vm[KS], vd[KS];
  {
    const int64_t r = (row0 + kj) * a.ld + kh * D + 8 * (lane >> 4);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      km[s] = *reinterpret_cast<const bf16x8_t*>(a.qkv_m + r + a.koff + 32 * s);
      kd[s] = *reinterpret_cast<const bf16x8_t*>(a.qkv_d + r + a.koff + 32 * s);
      vm[s] = *reinterpret_cast<const bf16x8_t*>(a.qkv_m + r + a.voff + 32 * s);
      vd[s] = *reinterpret_cast<const bf16x8_t*>(a.qkv_d + r + a.voff + 32 * s);
    }
  }
  // accumulators kt: keys k0 + 16 kt + 4 (lane / 16) + r, columns 16 wave + lane % 16
  f32x4_t Vm_[4], Vd_[4], Km_[4], Kd_[4];
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int r = 0; r < 4; ++r) Vm_[kt][r] = Vd_[kt][r] = Km_[kt][r] = Kd_[kt][r] = 0.f;

  const int nqb = (a.S - k0) / QB;   // query blocks from the first key on, per head
  const int total = nqb * a.G;
  auto issue = [&](int it) {
    const int g = it / nqb, qbk = it % nqb;
    const int h = kh * a.G + g, q0 = k0 + qbk * QB;
    const int64_t r = row0 + q0;
    const bf16_t* sq[2] = {a.qkv_m + r * a.ld + (int64_t)h * D, a.qkv_d + r * a.ld + (int64_t)h * D};
    const bf16_t* so[2] = {a.do_m + r * a.ldo + (int64_t)h * D, a.do_d + r * a.ldo + (int64_t)h * D};
    dma_tiles<D, QB, 2, 1, 8>(ring[it % 3], sq, a.ld, wave, lane);
    dma_tiles<D, QB, 2, 1, 8>(ring[it % 3] + 2 * TILE, so, a.ldo, wave, lane);
  };
  float4 nst = make_float4(0.f, 0.f, 0.f, 0.f);
  float ndd = 0.f;
  auto load_rows = [&](int it) {
    if (tid < QB) {
      const int g = it / nqb, qbk = it % nqb;
      const int64_t si = ((int64_t)b * a.Hq + kh * a.G + g) * a.S + k0 + qbk * QB + tid;
      const float4 st = a.stats[si];
      const float2 dl = a.delta[si];
      nst = make_float4(st.x, st.y, st.z, dl.x);
      ndd = dl.y;
    }
  };
  auto store_rows = [&](int it) {
    if (tid < QB) {
      sst[it & 1][tid] = nst;
      sdd[it & 1][tid] = ndd;
    }
  };
  load_rows(0);
  issue(0);
  __builtin_amdgcn_s_waitcnt(0);
  store_rows(0);
  __syncthreads();
  for (int it = 0; it < total; ++it) {
    if (it + 1 < total) {
      load_rows(it + 1);
      issue(it + 1);
    }
    const int q0 = k0 + (it % nqb) * QB;
    const bf16_t* Qm = ring[it % 3];
    bf16_t* pbuf = pbufs[it & 1];
    const bf16_t* Qd = Qm + TILE;
    const bf16_t* Om = Qm + 2 * TILE;
    const bf16_t* Od = Qm + 3 * TILE;
    {   // score phase: keys kw .. kw + 15, queries q0 + 16 qt .. + 15
      f32x4_t sm, sd, pm, pd;
#pragma unroll
      for (int r = 0; r < 4; ++r) sm[r] = sd[r] = pm[r] = pd[r] = 0.f;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const bf16x8_t qa = ld_k16<D>(Qm, 16 * qt, s, lane), qb_ = ld_k16<D>(Qd, 16 * qt, s, lane);
        sm = mma16(qa, km[s], sm);
        sd = mma16(qa, kd[s], sd);
        sd = mma16(qb_, km[s], sd);
        const bf16x8_t oa = ld_k16<D>(Om, 16 * qt, s, lane), ob = ld_k16<D>(Od, 16 * qt, s, lane);
        pm = mma16(oa, vm[s], pm);
        pd = mma16(oa, vd[s], pd);
        pd = mma16(ob, vm[s], pd);
      }
      float bmax = 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        sm[r] *= a.scale;
        sd[r] *= a.scale;
        bmax = fmaxf(bmax, fabsf(sd[r]));
      }
      if (q0 + 16 * qt < kw + 16) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (q0 + 16 * qt + 4 * (lane >> 4) + r < kj) sm[r] = NEG;
      }
      float Pm[4], Pd[4], gsm[4], gsd[4];
      auto terms = [&](auto ser) {
        const float4 ddv = *reinterpret_cast<const float4*>(&sdd[it & 1][16 * qt + 4 * (lane >> 4)]);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float4 st = sst[it & 1][16 * qt + 4 * (lane >> 4) + r];
          const float dd = r == 0 ? ddv.x : (r == 1 ? ddv.y : (r == 2 ? ddv.z : ddv.w));
          const float e = __expf(sm[r] - st.x);
          float c, sn;
          coshsinh<decltype(ser)::value>(sd[r], c, sn);
          const float P_m = e * (c * st.y - sn * st.z), P_d = e * (sn * st.y - c * st.z);
          const float xm = pm[r] - st.w, xd = pd[r] - dd;
          Pm[r] = P_m;
          Pd[r] = P_d;
          gsm[r] = P_m * xm + P_d * xd;
          gsd[r] = P_m * xd + P_d * xm;
        }
      };
      if (!__any(bmax >= SERIES_MAX)) terms(std::true_type{});
      else terms(std::false_type{});
      // lane (g, i) holds queries 16 qt + 4g .. + 3 of key 16 kg + i: half qt of slot g of that key row
      const int prow = 16 * kg + (lane & 15), g = lane >> 4, hf = 4 * (qt ^ ((g ^ (g >> 1)) & 1));
      *reinterpret_cast<v4i16*>(&pbuf[tswz<D, 2>(prow, g) + hf]) = pack4(Pm);
      *reinterpret_cast<v4i16*>(&pbuf[tswz<D, 2>(prow, 4 + g) + hf]) = pack4(Pd);
      *reinterpret_cast<v4i16*>(&pbuf[tswz<D, 2>(prow, 8 + g) + hf]) = pack4(gsm);
      *reinterpret_cast<v4i16*>(&pbuf[tswz<D, 2>(prow, 12 + g) + hf]) = pack4(gsd);
    }
    __builtin_amdgcn_s_waitcnt(0);   // own loads of the next block
    if (it + 1 < total) store_rows(it + 1);
    __syncthreads();   // every wavefront's P and dS are in the buffer, the next block is in the ring
    {   // dV, dK phase: all 64 keys, columns 16 wave .. + 15
      const int n0 = 16 * wave;
      const bf16x8_t om = ld_t16<D, true>(Om, 0, n0, lane), od = ld_t16<D, true>(Od, 0, n0, lane);
      const bf16x8_t qa = ld_t16<D, true>(Qm, 0, n0, lane), qb_ = ld_t16<D, true>(Qd, 0, n0, lane);
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        const bf16x8_t apm = ld_k16<D, 2>(pbuf, 16 * kt, 0, lane), apd = ld_k16<D, 2>(pbuf, 16 * kt, 1, lane);
        const bf16x8_t asm_ = ld_k16<D, 2>(pbuf, 16 * kt, 2, lane), asd = ld_k16<D, 2>(pbuf, 16 * kt, 3, lane);
        Vm_[kt] = mma16(apm, om, Vm_[kt]);
        Vd_[kt] = mma16(apm, od, Vd_[kt]);
        Vd_[kt] = mma16(apd, om, Vd_[kt]);
        Km_[kt] = mma16(asm_, qa, Km_[kt]);
        Kd_[kt] = mma16(asm_, qb_, Kd_[kt]);
        Kd_[kt] = mma16(asd, qa, Kd_[kt]);
      }
    }
  }

#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int key = k0 + 16 * kt + 4 * (lane >> 4) + r;
      const int64_t o = (row0 + key) * a.ldg + kh * D + 16 * wave + (lane & 15);
      a.g_m[o + a.koff] = Km_[kt][r] * a.scale;
      a.g_d[o + a.koff] = Kd_[kt][r] * a.scale;
      a.g_m[o + a.voff] = Vm_[kt][r];
      a.g_d[o + a.voff] = Vd_[kt][r];
    }
}

}  // namespace

bool flash_supported(int dh, int S) { return (dh == 64 || dh == 128) && S % 128 == 0; }

static FlashArgs with_constants(const FlashArgs& a0) {
  FlashArgs a = a0;
  const double sc = a.scale;
  a.c_exp = (float)(sc * 1.4426950408889634);
  a.c_cosh = (float)(0.5 * sc * sc);
  a.c_sinh = (float)(sc * sc * sc / 6.0);
  return a;
}

hipError_t launch_flash_fwd(const FlashArgs& a0, int B, hipStream_t s) {
  const FlashArgs a = with_constants(a0);
  if (a.D == 128) {
    dim3 g(a.S / 64, B * a.Hq);
    hipLaunchKernelGGL((flash_fwd16_kernel<128, 4>), g, dim3(256), 0, s, a);
  } else {
    dim3 g(a.S / 128, B * a.Hq);
    hipLaunchKernelGGL(flash_fwd_kernel<64>, g, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_flash_bwd(const FlashArgs& a0, int B, hipStream_t s) {
  const FlashArgs a = with_constants(a0);
  const int nrows = B * a.S * a.Hq;
  dim3 gd((nrows + 15) / 16);
  if (a.D == 128) hipLaunchKernelGGL(flash_delta_kernel<128>, gd, dim3(256), 0, s, a, nrows);
  else hipLaunchKernelGGL(flash_delta_kernel<64>, gd, dim3(256), 0, s, a, nrows);
  if (a.D == 128) {
    dim3 gq(a.S / 64, B * a.Hq);
    hipLaunchKernelGGL((flash_bwd_q16_kernel<128, 4>), gq, dim3(256), 0, s, a);
  } else {
    dim3 gq(a.S / 128, B * a.Hq);
    hipLaunchKernelGGL(flash_bwd_q_kernel<64>, gq, dim3(256), 0, s, a);
  }
  // dK/dV: 64 keys per workgroup; for D = 128 eight wavefronts share the
  // probabilities through LDS
  dim3 gk(a.S / 64, B * a.Hk);
  if (a.D == 128) hipLaunchKernelGGL(flash_bwd_kv8_kernel<128>, gk, dim3(512), 0, s, a);
  else hipLaunchKernelGGL(flash_bwd_kv_kernel<64>, gk, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace fdh
