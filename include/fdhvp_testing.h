/*
 * fdhvp_testing.h - testing hooks of libfdhvp (not needed to use the library).
 *
 * They expose internal kernels on caller-owned device buffers so that the test
 * suite can check each one in isolation against a plain host computation.
 */
#ifndef FDHVP_TESTING_H
#define FDHVP_TESTING_H

#include "fdhvp.h"

#ifdef __cplusplus
extern "C" {
#endif

/* The internal batched MFMA GEMM:
 *   C[z] = alpha * (A[z] B[z]^T + A2[z] B2[z]^T)        (second pair optional)
 * dtype: FDH_F32 (fp32 operands, v_mfma_f32_32x32x2_f32) or FDH_BF16 (uint16
 * bfloat16 operands, v_mfma_f32_32x32x16_bf16, fp32 accumulation).
 * A is [batch][M][K] when a_kmajor, else [batch][K][M]; B is [batch][N][K] when
 * b_kmajor, else [batch][K][N]; A2/B2 (may be NULL together) share the layouts.
 * C is float32 [batch][M][N], overwritten.  causal: 0 none, 1 skip output tiles
 * above the diagonal, 2 contract only k <= m, 3 only k >= m.  tile selects
 * the bf16 kernel variant (0 automatic, 1 128x128, 2 256x256, 3 256x128,
 * 4 256x256 and 5 256x128 fed by direct global-to-LDS loads, K % 32 == 0,
 * 6 as 4 with four 128x128 wavefront tiles instead of eight 128x64 ones,
 * 7 as 6 with 64-deep K slices in a two-stage ring, K % 64 == 0 and equal
 * operand strides in both pairs).
 * Enqueued on hip_stream; returns without waiting.  K, and M/N of MN-major
 * operands, must be multiples of 8 (bf16) or 4 (fp32). */
fdh_status fdh_testing_gemm(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t batch, int32_t a_kmajor,
                            int32_t b_kmajor, const void* A, const void* B, const void* A2, const void* B2,
                            float* C, int32_t causal, float alpha, int32_t tile, void* hip_stream);

/* Two independent bf16 products in one launch of the 256 x 256 kernel given
 * by tile (6 or 8, as for fdh_testing_gemm), the way the weight gradients of
 * the attention output and q/k/v projections share a launch in an HVP.
 * Product p is C_p[batch_p][M_p][N_p] = alpha (A_p B_p^T + A2_p B2_p^T) per
 * batch entry, operands laid out as for fdh_testing_gemm, both products with
 * the same a_kmajor / b_kmajor; A2_p, B2_p may be NULL together.  K_p % 32 ==
 * 0, M_p and N_p >= 8, batch_p >= 1.  FDH_ERR_UNSUPPORTED when a product does
 * not fit the kernel.  Enqueued on hip_stream; returns without waiting. */
fdh_status fdh_testing_gemm_pair(int32_t M0, int32_t N0, int32_t K0, int32_t batch0, int32_t M1, int32_t N1,
                                 int32_t K1, int32_t batch1, int32_t a_kmajor, int32_t b_kmajor, const void* A0,
                                 const void* B0, const void* A20, const void* B20, float* C0, const void* A1,
                                 const void* B1, const void* A21, const void* B21, float* C1, float alpha,
                                 int32_t tile, void* hip_stream);

/* on != 0 makes the next fdh_set_workspace plan the unfused attention path
 * (score, probability and score-gradient matrices in the workspace, MFMA
 * GEMMs and row kernels) even where the fused kernels apply (bf16 operands,
 * head dimension 64 or 128, S a multiple of 128), so that the two paths can
 * be compared on one model. */
fdh_status fdh_testing_unfused_attention(fdh_ctx* ctx, int32_t on);

/* Weight-gradient launch forms, so that they can be compared.  By default
 * (on = 0) small output grids are cut into token slices whose fp32 partial
 * products are added afterwards (fp64 sums in slice order), and with fused
 * attention the attention output projection's weight gradient shares one
 * launch with the q/k/v one when its tiles fit into that grid's last wave.
 * on = 1: every weight gradient contracts over the whole token range in a
 * launch of its own; on = 2: token slices as by default, no shared launch.
 * Other values: FDH_ERR_INVALID_ARG.  Takes effect at the next HVP. */
fdh_status fdh_testing_unsplit_wgrad(fdh_ctx* ctx, int32_t on);

/* Per-launch timing with HIP events recorded on the context stream around every
 * GEMM launch (category 0), every Lanczos vector launch (category 1) and every
 * fused attention forward and backward (category 2).
 * enable != 0 turns it on (and clears the accumulators).  While on, the event
 * pool is drained with a stream synchronisation every few thousand launches. */
fdh_status fdh_testing_timing(fdh_ctx* ctx, int32_t enable);
/* Waits for the stream, then writes for categories c = 0..3:
 * out[4c+0] launches, out[4c+1] summed milliseconds, out[4c+2] executed FLOPs
 * (GEMM: 2*rows*cols*k per tile, tails clipped; attention: algorithmic causal
 * products of both passes, without the backward's score recompute), out[4c+3] algorithmic bytes
 * (Lanczos: every operand read or written once).  Clears the accumulators. */
fdh_status fdh_testing_timing_read(fdh_ctx* ctx, double* out16);

/* Digest (FNV-1a) of the workspace carve the context has adopted: every
 * buffer's offset and size, the basis geometry, the attention path, the plan
 * and the workspace pointer.  Host-only; lets tests check that size queries
 * and rejected fdh_set_workspace calls leave the carve in use untouched. */
fdh_status fdh_testing_layout_digest(const fdh_ctx* ctx, uint64_t* out);

/* Plain device copy of `bytes` bytes (16-byte vectors), enqueued on hip_stream;
 * used to calibrate hardware byte counters against a known traffic. */
fdh_status fdh_testing_copy(void* dst, const void* src, size_t bytes, void* hip_stream);

#ifdef __cplusplus
}
#endif
#endif /* FDHVP_TESTING_H */
