// Launchers for the HIP kernels (internal interface between the host engine and
// the device code).  Every launcher enqueues on the given stream and returns
// the launch status; none synchronises.
#pragma once
#include "common.h"
#include "gemm.h"

namespace fdh {

// SplitMix64 streams (one per purpose)
constexpr uint64_t STREAM_PARAMS = 1, STREAM_TOKENS = 2, STREAM_PROBE = 3, STREAM_GAUSS = 4;

// ---- rng.hip ---------------------------------------------------------------
template <typename T>
hipError_t launch_init_range(T* theta, int64_t off, int64_t n, int kind, uint64_t seed, double stdv, hipStream_t s);
hipError_t launch_tokens_uniform(int32_t* tok, int64_t n, uint64_t seed, int V, hipStream_t s);
hipError_t launch_tokens_zipf(int32_t* tok, int64_t n, uint64_t seed, const double* cdf, int V, hipStream_t s);
hipError_t launch_rademacher(float* out, int64_t n, uint64_t seed, hipStream_t s);
hipError_t launch_gaussian_unit(float* out, double* partial1024, int64_t n, uint64_t seed, hipStream_t s);

// ---- vec.hip ---------------------------------------------------------------
constexpr int RED_BLOCKS = 1024;   // fixed grid of the deterministic reductions

hipError_t launch_fill_f32(float* p, int64_t n, float v, hipStream_t s);
hipError_t launch_copy16(void* dst, const void* src, size_t bytes, hipStream_t s);
hipError_t launch_fill_f64(double* p, int64_t n, double v, hipStream_t s);
// out[i] = sum_{j < ns} part[j * n + i] (acc: out[i] += that sum), summed in fp64
// in the order j = 0, 1, ...
hipError_t launch_sum_splits(float* out, const float* part, int ns, int64_t n, bool acc, hipStream_t s);
// lo[i] = T(eps * v[i])
template <typename T>
hipError_t launch_scale_cast(T* lo, const float* v, double eps, int64_t n, hipStream_t s, int* nonfinite = nullptr);
// nonfinite[0] = 1 when some x[i], i < n, is NaN or infinite (left alone otherwise)
hipError_t launch_nonfinite_scan(const float* x, int64_t n, int* flag, hipStream_t s);
// QUAD_DIAG: hv = (d (theta + eps v) - d (theta - eps v)) / (2 eps), both points in fp64
template <typename T>
hipError_t launch_quad_diag_hvp(const T* theta, const float* d, const float* v, double eps, float* hv, int64_t n, hipStream_t s);

// Lanczos state kept in device memory (fp64 scalars)
struct LanczosDev {
  double* alpha;     // [m]
  double* beta;      // [m]  beta[k] = beta_{k+2} in 1-based notation (residual after step k)
  double* coef;      // [128] reorthogonalisation coefficients of the current step
  double* gram;      // [128 * 128] Gram matrix Q^T Q of the stored basis rows (by slot)
  double* partial;   // [RED_BLOCKS * (2 * cap + 1)]
  int* flag;         // [2]: [0] = breakdown step + 1 (0 = none), [1] = spare
  double* maxabs;    // [1]  max_j |alpha_j| so far
};

// The stored Krylov rows, ldq elements apart (a multiple of 8): rows
// [0, ndev) in device memory at dev, rows [ndev, cap) at host, a device-side
// address of pinned host memory (the basis offload), read over the host link.
template <typename B>
struct BasisRows {
  B* dev = nullptr;
  B* host = nullptr;
  int ndev = 0;
  int64_t ldq = 0;
  __host__ __device__ B* row(int j) const {
    return j < ndev ? dev + (int64_t)j * ldq : host + (int64_t)(j - ndev) * ldq;
  }
};

// One Lanczos step after w = H q_k:
// Step A:  w <- w - beta_{k-1} q_prev;  alpha_k = <w, q>  (beta_{-1} = 0)
hipError_t launch_lanczos_alpha(float* w, const float* q, const float* qprev, LanczosDev st, int k, int64_t n, hipStream_t s);
// Step B (nv >= 1 stored rows, slot `newest` holds q_k), with step A fused:
// w' = w - beta_{k-1} q_prev (formed, not stored), alpha_k = <w', q>,
// p = Q^T w' - alpha_k g and g = Q^T Q_newest; alpha[k] written; Gram
// row/column `newest` <- g; coef = 2 p - G p (both classical Gram-Schmidt passes).
template <typename B>
hipError_t launch_lanczos_project(const float* w, const float* q, const float* qprev, BasisRows<B> rows, int nv, int newest,
                                  LanczosDev st, int k, int64_t n, hipStream_t s);
// Step C:  w <- (w' - alpha_k q) - Q coef (no rows when nv == 0); then ||w||^2.
// w' = w - beta_{k-1} qprev when qprev is given (step A fused into step B),
// else w itself (step A ran and stored it).
template <typename B>
hipError_t launch_lanczos_update(float* w, const float* q, const float* qprev, BasisRows<B> rows, int nv, LanczosDev st,
                                 int k, int64_t n, hipStream_t s);
// Step D:  beta_k = ||w||; breakdown test (tol relative to max |alpha|);
// q_next = w / beta_k; basis row (if not null) = B(q_next); the next HVP's
// perturbation operand (if lo is not null) = T(eps * q_next).
template <typename B, typename T>
hipError_t launch_lanczos_normalise(const float* w, float* qnext, B* basis_row, T* lo, double eps, LanczosDev st, int k, double tol,
                                    int64_t n, hipStream_t s);

// Conjugate gradient for (H + lam I) x = b: device scalars sc[5] = (r, r),
// (p, A p), alpha, (r_new, r_new), beta; partial: [RED_BLOCKS].
// init: x = 0, r = p = b, sc[0] = (b, b)
hipError_t launch_cg_init(float* x, float* r, float* p, const float* b, double* sc, double* partial, int64_t n,
                          hipStream_t s);
// ap <- ap + lam p (ap holds H p); sc[1] = (p, A p), sc[2] = alpha (0 unless (p, A p) > 0)
hipError_t launch_cg_ap(float* ap, const float* p, double lam, double* sc, double* partial, int64_t n, hipStream_t s);
// x += alpha p, r -= alpha A p; sc[3] = (r, r), sc[4] = beta, sc[0] = (r, r)
hipError_t launch_cg_step(float* x, float* r, const float* p, const float* ap, double* sc, double* partial, int64_t n,
                          hipStream_t s);
// p = r + beta p; lo (if not null) = T(eps p)
template <typename T>
hipError_t launch_cg_dir(float* p, const float* r, const double* sc, T* lo, double eps, int64_t n, hipStream_t s);

// Per-block sums over host ranges [nblk][2]:
// out[b*4 + {0,1,2,3}] = ||a_b||^2, ||b_b||^2, <a_b, b_b>, ||a_b - b_b||^2
hipError_t launch_block_stats(const float* a, const float* b, const int64_t* ranges, int nblk, double* partial, double* out, hipStream_t s);
// out = v on [s0, s1), 0 elsewhere (length n)
hipError_t launch_mask_range(float* out, const float* v, int64_t s0, int64_t s1, int64_t n, hipStream_t s);

// ---- lm.hip ----------------------------------------------------------------
// All "pair" tensors are two buffers: m (mean of the two points) and d (half difference).
struct PairF { float* m; float* d; };
template <typename T> struct PairT { T* m; T* d; };

template <typename T>
hipError_t launch_cast_pair(PairT<T> out, const float* m, const float* d, int64_t n, hipStream_t s);

// x = E[tok] (+ Pos[s]);  m = theta rows, d = eps * v rows; bad_tok[0] = 1
// (when bad_tok is not null) if a token lies outside [0, V) (it is clamped)
template <typename T>
hipError_t launch_embed_fwd(PairF x, const int32_t* tok, int T_, int S, int dmodel, int V,
                            const T* th_e, const float* v_e, const T* th_p, const float* v_p, double eps, int* bad_tok,
                            hipStream_t s);

// Norm forward at both points: y = norm(x; g +- eps vg, b +- eps vb)
template <typename T>
hipError_t launch_norm_fwd(PairT<T> y, const float* xm, const float* xd, int rows, int dmodel, bool layernorm,
                           const T* th_g, const float* v_g, const T* th_b, const float* v_b, double eps, float norm_eps, hipStream_t s);
// Norm backward at both points: dx_out = dx_res + d/dx, and dx_op (if dx_op.m is
// not null) = the operand-type copy of dx_out.  Rows are taken norm_bwd_groups(rows)
// workgroups at a time: gpart[w][j] (fp64) = the workgroup's sum over its rows
// of the half difference of dy * xhat (gain gradient), and with bpart (LayerNorm)
// bpart[w][j] = its sum of dy.d (bias gradient); launch_colsum_f64 finishes both.
// dmodel * (bpart ? 2 : 1) <= 8192.
constexpr int NORM_BWD_ROWS = 16;
inline int norm_bwd_groups(int rows) { return (rows + NORM_BWD_ROWS - 1) / NORM_BWD_ROWS; }
template <typename T>
hipError_t launch_norm_bwd(PairF dx_out, PairT<T> dx_op, const float* dres_m, const float* dres_d, const float* xm,
                           const float* xd, const float* dym, const float* dyd, int rows, int dmodel, bool layernorm,
                           const T* th_g, const float* v_g, double eps, float norm_eps, double* gpart, double* bpart,
                           hipStream_t s);

// out[j] = scale * sum_t X[t*ld + j] (deterministic); accumulate adds to out.  partial: [64 * C]
hipError_t launch_colsum(float* out, const float* X, int rows, int C, int64_t ld, double scale, bool accumulate,
                         double* partial, hipStream_t s);
// the same for fp64 rows X [rows][C]
hipError_t launch_colsum_f64(float* out, const double* X, int rows, int C, double scale, bool accumulate, double* partial,
                             hipStream_t s);

// RoPE (Llama) of the q and k columns, in place on both channels of the
// operand-type projection output [T, (Hq + 2 Hk) dh]; v is left as it is
template <typename T>
hipError_t launch_rope_inplace(PairT<T> qkv, int T_, int S, int Hq, int Hk, int dh, const double* cs, hipStream_t s);
// backward RoPE on dq/dk columns (fp32, in place) + cast of dq,dk,dv into operand type
template <typename T>
hipError_t launch_qkv_bwd_post(PairT<T> out, float* gm, float* gd, int T_, int S, int Hq, int Hk, int dh,
                               const double* rope_cs, bool rope, hipStream_t s);
// rope table: cs[s*dh + 2i] = cos(s * base^(-2i/dh)), cs[s*dh + 2i + 1] = sin(...)
hipError_t launch_rope_table(double* cs, int S, int dh, double base, hipStream_t s);

// causal softmax at both points: rows of S scores (fp32 pairs, already scaled) -> P (operand type)
template <typename T>
hipError_t launch_attn_softmax(PairT<T> P, const float* Sm, const float* Sd, int nrows_total, int S, hipStream_t s);
// dS = P (dP - rowsum(P dP)) at both points
template <typename T>
hipError_t launch_attn_dsoftmax(PairT<T> dS, const T* Pm, const T* Pd, const float* dPm, const float* dPd,
                                int nrows_total, int S, hipStream_t s);
// GQA: sum groups of G consecutive query-head gradients into KV heads
hipError_t launch_group_sum(float* out, int64_t out_ld, const float* in, int T_, int Hk, int G, int dh, hipStream_t s);

// ---- attn.hip: fused causal attention of the pair (bf16 operands) ------------
struct FlashArgs {
  const bf16_t* qkv_m;   // [T][ld]: post-RoPE q (cols h*D), k (koff + kh*D), v (voff + kh*D)
  const bf16_t* qkv_d;
  int64_t ld;
  int S, Hq, Hk, G, D;   // G = Hq / Hk query heads per key/value head
  int koff, voff;
  float scale;           // 1 / sqrt(D)
  bf16_t* o_m;           // [T][ldo] attention output (forward), input of the backward
  bf16_t* o_d;
  int64_t ldo;
  float4* stats;         // [B*Hq][S]: row max of the logits, u, w (forward -> backward)
  const bf16_t* do_m;    // [T][ldo] output gradient (backward)
  const bf16_t* do_d;
  float2* delta;         // [B*Hq][S] row terms (backward scratch)
  float* g_m;            // [T][ldg] fp32 gradients of q, k, v (same column layout as qkv)
  float* g_d;
  int64_t ldg;
  // derived from scale by the launchers: scale log2(e), scale^2 / 2, scale^3 / 6
  float c_exp, c_cosh, c_sinh;
};
// head dimension 64 or 128, S a multiple of 128
bool flash_supported(int dh, int S);
hipError_t launch_flash_fwd(const FlashArgs& a, int B, hipStream_t s);
// row terms, dq (query columns of g) and dk, dv (key/value columns, summed over each group)
hipError_t launch_flash_bwd(const FlashArgs& a, int B, hipStream_t s);

// activations at both points
template <typename T>
hipError_t launch_gelu_fwd(PairT<T> z, const T* um, const T* ud, int64_t n, hipStream_t s);
template <typename T>
hipError_t launch_gelu_bwd(PairT<T> du, float* dud_f32, const T* um, const T* ud, const float* dzm, const float* dzd,
                           int64_t n, hipStream_t s);
template <typename T>
hipError_t launch_swiglu_fwd(PairT<T> z, const T* gum, const T* gud, int rows, int F, hipStream_t s);
template <typename T>
hipError_t launch_swiglu_bwd(PairT<T> dgu, const T* gum, const T* gud, const float* dzm, const float* dzd,
                             int rows, int F, hipStream_t s);

// cross-entropy at both points: dlogits (operand type) and per-row losses (fp64, [2][T]),
// every kept row scaled by inv_n; targets from lab (int32 [B, S], IGNORE_LABEL
// drops a target) or, with lab == nullptr, the next token
constexpr int IGNORE_LABEL = -100;
template <typename T>
hipError_t launch_ce(PairT<T> dl, double* rowloss, const float* lm, const float* ld, const int32_t* tok,
                     const int32_t* lab, int T_, int S, int V, double inv_n, hipStream_t s);
// out2 = (or += with acc) the sums of the two rows of rowloss
hipError_t launch_loss_sum(double* out2, const double* rowloss, int T_, bool acc, hipStream_t s);
// out3[0] += targets of a [B, S] batch, out3[1] += labels outside [0, V) other
// than IGNORE_LABEL (lab may be null: next-token targets), out3[2] += tokens outside [0, V)
hipError_t launch_count_targets(int64_t* out3, const int32_t* tok, const int32_t* lab, int B, int S, int V, hipStream_t s);

// embedding backward (difference channel only): deterministic sort + segment sums
hipError_t launch_token_sort(uint32_t* keys, const int32_t* tok, int T_, int V, hipStream_t s);
hipError_t launch_embed_bwd(float* hv_e, const uint32_t* keys, const float* dxd, int T_, int dmodel, double inv_eps,
                            bool accumulate, hipStream_t s);
hipError_t launch_pos_bwd(float* hv_p, const float* dxd, int B, int S, int dmodel, double inv_eps, bool accumulate,
                          hipStream_t s);

}  // namespace fdh
