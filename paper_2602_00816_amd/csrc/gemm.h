// Batched MFMA GEMM with operand pairs:  C[z] = alpha * sum_p A_p[z] B_p[z]^T (+ epilogue)
#pragma once
#include "common.h"

namespace fdh {

enum GemmOut { OUT_F32 = 0, OUT_OP = 1 };
enum GemmCausal {
  CAUSAL_NONE = 0,
  CAUSAL_SKIP_UPPER = 1,  // output tiles strictly above the diagonal (n > m) are not computed
  CAUSAL_K_LE_M = 2,      // contraction restricted to k <= m (rows of a lower-triangular A)
  CAUSAL_K_GE_M = 3       // contraction restricted to k >= m (rows of an upper-triangular A)
};

// Element (r, k) of an operand lives at ptr + off(z) + r*s_row + k*s_k, with
// exactly one of s_row, s_k equal to 1 ("K-major" when s_k == 1, "MN-major"
// when s_row == 1).  off(z) = (z / inner_count)*s_outer + ((z % inner_count) / inner_div)*s_inner.
struct GemmOperand {
  const void* ptr = nullptr;
  int64_t s_row = 0, s_k = 1;
  int64_t s_outer = 0, s_inner = 0;
  int32_t inner_div = 1;
};

struct GemmArgs {
  int M = 0, N = 0, K = 0;
  int nbatch = 1, inner_count = 1;
  int npairs = 1;
  GemmOperand A[2], B[2];
  void* C = nullptr;
  int64_t ldc = 0, c_outer = 0, c_inner = 0;
  int32_t c_div = 1;
  int out_type = OUT_F32;
  float alpha = 1.f, beta = 0.f;          // C = alpha*acc + beta*C_old (beta only with OUT_F32)
  const void* bias_theta = nullptr;       // operand-type vector [N], added times bias_theta_scale
  float bias_theta_scale = 1.f;
  const float* bias_v = nullptr;          // float vector [N], added times bias_v_scale
  float bias_v_scale = 1.f;
  const float* resid = nullptr;           // fp32, same indexing as C, added (OUT_F32 only)
  int causal = CAUSAL_NONE;
  int tile = 0;                           // 0 automatic; bf16 only: 1 128x128, 2 256x256, 3 256x128
};

// T = float (fp32 MFMA) or bf16_t (bf16 MFMA, fp32 accumulation)
template <typename T>
hipError_t gemm(const GemmArgs& a, hipStream_t stream);

// Two independent products (batched or not, no causal limits) in one launch
// of the 256 x 256 kernel that a0 runs on, when a1 can run on it too; else one
// launch each.  Each output gets the same arithmetic as in a launch of its own
// on that kernel.
template <typename T>
hipError_t gemm_pair(const GemmArgs& a0, const GemmArgs& a1, hipStream_t stream);

// Host-side validation of the shapes, strides and alignment the kernel assumes.
// Returns nullptr if fine, else a message.
template <typename T>
const char* gemm_check(const GemmArgs& a);

}  // namespace fdh
