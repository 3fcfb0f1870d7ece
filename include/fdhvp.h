/*
 * fdhvp.h - finite-difference Hessian-vector products, Lanczos and stochastic
 * Lanczos quadrature for decoder-only language-model losses on AMD MI355X
 * (gfx950).  C ABI: plain pointers and sizes, no framework types.
 *
 * The operation (section 3.1, Eq. grad-fd-hvp; Algorithm 1): for parameters
 * theta, a direction v and a step eps,
 *     Hv ~= (grad L(theta + eps v) - grad L(theta - eps v)) / (2 eps),
 * where L is the mean next-token cross-entropy of the model over one token
 * batch.  Lanczos (section 4; Appendix C) drives it to build the tridiagonal
 * T_m = (alpha, beta); SLQ (section 4) turns T_m into Gauss quadrature nodes
 * (Ritz values) and weights.
 *
 * Conventions shared by every call
 *  - Ownership: the caller owns every buffer.  Device pointers: parameters,
 *    directions, outputs, tokens and the workspace.  Host pointers: alpha,
 *    beta, nodes, weights, statistics.  The library never allocates device
 *    memory; it carves all scratch from the workspace given to
 *    fdh_set_workspace.
 *  - Parameter vector: one flat array in the order reported by
 *    fdh_param_layout (per-layer blocks contiguous).  Element type float32
 *    (dtype FDH_F32) or bfloat16 bit patterns, uint16 (FDH_BF16).  Directions
 *    v and products Hv are always float32 of length fdh_num_params().
 *  - Tokens: int32 [B, S] row-major, values in [0, vocab); a token outside
 *    that range is an FDH_ERR_INVALID_ARG (never clamped into a wrong answer).
 *  - Streams: all device work is enqueued on the stream given to fdh_create,
 *    in call order.  fdh_hvp and fdh_hvp_bound wait for the stream at their
 *    end, to report non-finite values and bad tokens; so do the calls that
 *    return host results (lanczos, slq_density, block_stats, last_losses,
 *    the binds, cg_solve, block_diagonal).
 *  - Errors: every call returns an fdh_status; negative values are errors and
 *    leave outputs unspecified; fdh_last_error gives a message.  No call
 *    throws.  One context per host thread.
 *  - theta is never written: the perturbed points are formed on the fly.
 */
#ifndef FDHVP_H
#define FDHVP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FDH_API_VERSION 1

typedef enum fdh_status {
  FDH_OK = 0,
  FDH_BREAKDOWN = 1,          /* warning: Lanczos stopped early, see steps_done */
  FDH_ERR_INVALID_ARG = -1,   /* null pointer, bad size/shape, eps <= 0 or not finite, m < 1 */
  FDH_ERR_WORKSPACE = -2,     /* no workspace, or smaller than fdh_workspace_bytes */
  FDH_ERR_HIP = -3,           /* a HIP runtime call failed */
  FDH_ERR_NONFINITE = -4,     /* NaN/Inf found in an input direction or in a product */
  FDH_ERR_STATE = -5,         /* call order (e.g. lanczos before bind) */
  FDH_ERR_UNSUPPORTED = -6    /* configuration outside what the kernels support */
} fdh_status;

typedef enum fdh_family {
  FDH_FAMILY_GPT2 = 0,        /* LayerNorm, learned positions, GELU(tanh) MLP, biases, tied head */
  FDH_FAMILY_LLAMA = 1,       /* RMSNorm, RoPE, SwiGLU MLP, GQA, no biases, untied head */
  FDH_FAMILY_QUAD_DIAG = 2    /* L(theta) = 1/2 sum_i d_i theta_i^2 (test operator, Hv = d*v) */
} fdh_family;

typedef enum fdh_dtype { FDH_F32 = 0, FDH_BF16 = 1 } fdh_dtype;
typedef enum fdh_reorth { FDH_REORTH_NONE = 0, FDH_REORTH_FULL = 1, FDH_REORTH_WINDOW = 2 } fdh_reorth;
typedef enum fdh_token_dist { FDH_TOKENS_UNIFORM = 0, FDH_TOKENS_ZIPF = 1 } fdh_token_dist;
typedef enum fdh_vec_kind { FDH_VEC_RADEMACHER = 0, FDH_VEC_GAUSSIAN = 1 } fdh_vec_kind;
typedef enum fdh_param_kind { FDH_PARAM_MATRIX = 0, FDH_PARAM_GAIN = 1, FDH_PARAM_BIAS = 2 } fdh_param_kind;

/* Model description.  For FDH_FAMILY_QUAD_DIAG only quad_n and dtype are read. */
typedef struct fdh_model_config {
  int32_t family;       /* fdh_family */
  int32_t n_layers;
  int32_t d_model;
  int32_t n_heads;
  int32_t n_kv_heads;   /* must divide n_heads */
  int32_t d_ff;
  int32_t vocab;
  int32_t max_seq;      /* learned-position rows (GPT-2) and upper bound on S */
  int32_t dtype;        /* fdh_dtype of the parameter vector and of the GEMM operands */
  float norm_eps;       /* LayerNorm / RMSNorm epsilon */
  float rope_base;      /* RoPE base (Llama family) */
  int32_t reserved;
  int64_t quad_n;       /* QUAD_DIAG dimension */
} fdh_model_config;

typedef struct fdh_lanczos_opts {
  int32_t reorth;       /* fdh_reorth */
  int32_t window;       /* WINDOW: number of most recent Lanczos vectors kept (>= 1) */
  int32_t basis_dtype;  /* fdh_dtype of the stored Krylov basis */
  float breakdown_tol;  /* stop when beta_{k+1} <= tol * max_j |alpha_j|; 0 selects 1e-5 */
} fdh_lanczos_opts;

/* Reduction of the per-target losses over a bound dataset. */
typedef enum fdh_reduction {
  FDH_REDUCE_MEAN = 0,        /* token-weighted mean over every kept target of every batch */
  FDH_REDUCE_SUM = 1          /* their sum (the solution-token objective of section 7) */
} fdh_reduction;

/* One batch of a dataset (Algorithm 1's dataloader): device pointers, caller-owned. */
typedef struct fdh_batch {
  const int32_t* tokens;  /* int32 [B, S] input tokens */
  const int32_t* labels;  /* int32 [B, S] aligned with the tokens: the logits at position t
                           * are scored against labels[t + 1]; -100 drops that target
                           * (padding, masked prompt).  NULL: the next token is the target. */
  int32_t B, S;
} fdh_batch;

typedef struct fdh_block {
  char name[48];        /* e.g. "h3.wqkv" */
  int64_t offset;       /* element offset in the flat vector */
  int64_t numel;
  int64_t rows, cols;   /* matrix shape (cols = 1 for vectors) */
  int32_t layer;        /* transformer layer, -1 for embeddings / final norm / head */
  int32_t kind;         /* fdh_param_kind */
} fdh_block;

typedef struct fdh_ctx fdh_ctx;

/* Create a context for one model on the current HIP device; hip_stream is a
 * hipStream_t (NULL = default stream).  *out receives the context. */
fdh_status fdh_create(const fdh_model_config* cfg, void* hip_stream, fdh_ctx** out);
void fdh_destroy(fdh_ctx* ctx);
int32_t fdh_api_version(void);

/* Number of parameters P (the length of theta, v and Hv). */
int64_t fdh_num_params(const fdh_ctx* ctx);

/* Parameter layout: up to cap entries into out; *n receives the total count. */
fdh_status fdh_param_layout(const fdh_ctx* ctx, fdh_block* out, int32_t cap, int32_t* n);

/* Workspace needed for token batches up to [B, S] and Lanczos runs up to m steps
 * with options o (o may be NULL and m 0 when only fdh_hvp is used). */
fdh_status fdh_workspace_bytes(const fdh_ctx* ctx, int32_t B, int32_t S, int32_t m,
                               const fdh_lanczos_opts* o, size_t* bytes);
/* Hand the library a device buffer of at least the queried size, 256-byte aligned.
 * The caller keeps ownership and must keep it alive while the context uses it.
 * On an error the workspace and carve already in use stay in force.  dev = NULL
 * with bytes = 0 detaches the workspace (the other arguments are ignored): the
 * context then holds no pointer into caller memory until the next call. */
fdh_status fdh_set_workspace(fdh_ctx* ctx, void* dev, size_t bytes, int32_t B, int32_t S,
                             int32_t m, const fdh_lanczos_opts* o);

/* Activation recomputation (gradient checkpointing, an option of the
 * fine-tuning runs of section 6): with on != 0 the workspace keeps, per
 * decoder layer, only the fp32 input pair of the layer (mean and
 * half-difference channels) plus one set of the layer's other activations
 * that all layers share.  Before each layer's backward the HVP runs that
 * layer's forward again from its stored input, up to the MLP activation, so
 * one HVP executes every decoder layer but the last one's forward twice (about
 * a quarter more GEMM work) and needs L - 1 fewer activation sets.  Results are the
 * same bits as without.  Takes effect for the following fdh_workspace_bytes /
 * fdh_set_workspace; the carve in use keeps its mode until then.  Off by
 * default; no effect for QUAD_DIAG. */
fdh_status fdh_set_recompute(fdh_ctx* ctx, int32_t on);

/* Synthetic inputs (the SplitMix64 counter generator of Steele, Lea and Flood,
 * OOPSLA 2014, in counter form): theta with N(0, 0.02) matrices, unit gains, zero biases (bf16 by
 * round-to-nearest-even); tokens uniform or Zipf(1.1); unit vectors. */
fdh_status fdh_init_params(fdh_ctx* ctx, void* params_dev, uint64_t seed);
fdh_status fdh_make_tokens(fdh_ctx* ctx, int32_t* tokens_dev, int32_t B, int32_t S,
                           uint64_t seed, int32_t dist);
fdh_status fdh_random_vector(fdh_ctx* ctx, float* out_dev, uint64_t seed, int32_t kind);

/* QUAD_DIAG only: the diagonal d (float32, length P, device, caller-owned). */
fdh_status fdh_set_quad_diag(fdh_ctx* ctx, const float* diag_dev);

/* Hv ~= (grad L(theta + eps v) - grad L(theta - eps v)) / (2 eps) on one batch
 * (section 3.1; Algorithm 1 with a single batch).  params: P elements of the
 * context dtype; v, hv: float32 [P]; tokens int32 [B, S] (ignored for QUAD_DIAG).
 * hv must not alias params or v.  Waits for the stream before returning.
 * Language-model families: FDH_ERR_NONFINITE when v holds a NaN or an
 * infinity, or when the product does (both scanned on the device, one extra
 * read of Hv); FDH_ERR_INVALID_ARG when a token lies outside [0, vocab).  On
 * either error hv is unspecified.  (QUAD_DIAG, a test operator, is not scanned.) */
fdh_status fdh_hvp(fdh_ctx* ctx, const void* params_dev, const float* v_dev, double eps,
                   const int32_t* tokens_dev, int32_t B, int32_t S, float* hv_dev);

/* Loss values L(theta + eps v), L(theta - eps v) of the most recent fdh_hvp. */
fdh_status fdh_last_losses(fdh_ctx* ctx, double* loss_plus, double* loss_minus);

/* Fix the operator used by fdh_hvp_bound / fdh_lanczos / fdh_slq_density /
 * fdh_cg_solve / fdh_block_diagonal: one batch of next-token targets (the same
 * as fdh_bind_dataset with one unlabelled batch and FDH_REDUCE_MEAN, whose
 * token scan and wait it shares).  The pointers are kept (not copied) and must
 * stay valid. */
fdh_status fdh_bind(fdh_ctx* ctx, const void* params_dev, const int32_t* tokens_dev,
                    int32_t B, int32_t S, double eps);

/* Fix a dataset operator for fdh_hvp_bound / fdh_lanczos / fdh_slq_density /
 * fdh_cg_solve / fdh_block_diagonal (Algorithm 1 with its dataloader loop,
 * section 3.1): the FD-HVP of the loss over all nbatch batches, each batch
 * weighted by its number of kept targets w_b, so that with FDH_REDUCE_MEAN
 * the result is the HVP of the token-weighted mean loss
 * sum_b w_b L_b / sum_b w_b (L_b the mean over batch b's targets), and with
 * FDH_REDUCE_SUM that of the summed loss.  Batches may differ in B and S,
 * each within the workspace plan (and S a multiple of 128 where the plan uses
 * fused attention).  Padding is taken to sit after the real tokens (right
 * padding) with label -100: causal attention then keeps it out of every kept
 * target's context, so no attention mask is needed.  The batch array is
 * copied, the device pointers are kept (not copied) and must stay valid.
 * *n_targets (may be NULL) receives sum_b w_b.  Tokens and labels are scanned
 * on the device and the call waits for the stream; FDH_ERR_INVALID_ARG for a
 * token outside [0, vocab), a label outside [0, vocab) other than -100, or
 * when no target is left.
 * QUAD_DIAG contexts take nbatch = 0. */
fdh_status fdh_bind_dataset(fdh_ctx* ctx, const void* params_dev, const fdh_batch* batches, int32_t nbatch,
                            double eps, int32_t reduction, int64_t* n_targets);

/* hv = H v of the bound operator (fdh_bind or fdh_bind_dataset): one FD-HVP
 * per batch, accumulated into hv in batch order; fdh_last_losses then returns
 * the dataset losses at theta +- eps v.  v, hv: float32 [P] on device, not
 * aliasing each other or the parameters.  Waits for the stream and reports
 * non-finite values and bad tokens as fdh_hvp does. */
fdh_status fdh_hvp_bound(fdh_ctx* ctx, const float* v_dev, float* hv_dev);

/* Krylov-basis offload (section 7 notes that storing the whole Krylov
 * subspace bounds the scale and names offloading part of it to host memory):
 * keep at most device_rows stored Lanczos rows in the workspace and the
 * remaining ones in host_rows, caller-owned pinned host memory mapped for the
 * device (hipHostMalloc), of at least (stored rows - device_rows) * row bytes,
 * where stored rows = m (full) or min(m, window) and row bytes =
 * round_up(P, 8) * (2 for a bf16 basis, 4 for fp32).  Takes effect for the
 * following fdh_workspace_bytes / fdh_set_workspace (the workspace then holds
 * device_rows rows) and Lanczos runs; device_rows < 0 keeps every row on the
 * device (the default) and forgets host_rows.  The projection and update
 * passes read the host rows over the host link at every step, so each host
 * row adds about 2 * row bytes / link bandwidth to a step; results are the
 * same bits as with every row on the device.  FDH_ERR_INVALID_ARG when
 * host_rows is not mapped pinned memory or device_rows > 128; a Lanczos run
 * whose host part does not fit host_bytes fails with FDH_ERR_WORKSPACE. */
fdh_status fdh_set_basis_offload(fdh_ctx* ctx, int32_t device_rows, void* host_rows, size_t host_bytes);

/* m Lanczos steps (section 4) from the Rademacher probe z/sqrt(P) drawn from
 * probe_seed.  alpha_host[m], beta_host[m] receive alpha_1..alpha_s and
 * beta_2..beta_{s+1} (the last is the residual norm), s = *steps_done <= m;
 * entries past s are zero.  Returns FDH_BREAKDOWN when s < m. */
fdh_status fdh_lanczos(fdh_ctx* ctx, int32_t m, uint64_t probe_seed, const fdh_lanczos_opts* o,
                       double* alpha_host, double* beta_host, int32_t* steps_done);

/* SLQ (section 4): for probe j = 0..probes-1, Lanczos from seed + j, then the
 * eigen-decomposition of T_s: nodes_host[j*m + i] = lambda_i, weights_host[j*m+i]
 * = (U_1i)^2 (zero-padded past steps_done[j]); *trace_est = P * mean_j alpha_1. */
fdh_status fdh_slq_density(fdh_ctx* ctx, int32_t probes, int32_t m, uint64_t seed,
                           const fdh_lanczos_opts* o, double* nodes_host, double* weights_host,
                           int32_t* steps_done, double* trace_est);

/* Ritz-value diagnostics for runs that lose orthogonality (no or windowed
 * reorthogonalisation; Theorem 4.1's spurious duplicate "ghost" eigenvalues).
 * Host-only, no context.  alpha[s], beta[s] as returned by fdh_lanczos
 * (beta[s - 1] = beta_{s+1} is the residual norm), 1 <= s <= 128.  With
 * norm = max_i |theta_i| over the Ritz values theta_i of T_s (ascending):
 * nodes[i] = theta_i; weights[i] = (U_1i)^2; resid[i] = beta_{s+1} |U_si|,
 * the residual norm of the Ritz pair while the basis stays orthonormal;
 * copies[i] = size of its cluster (Ritz values chained by gaps <= tol * norm);
 * spurious[i] = 1 for a simple Ritz value that is also an eigenvalue of T_s
 * without its first row and column, within tol * norm (the test of Cullum and
 * Willoughby, 1985); *n_ghosts = sum over clusters of (size - 1).  Any output
 * pointer may be NULL.  FDH_ERR_INVALID_ARG for s outside [1, 128], a null
 * input or tol < 0. */
fdh_status fdh_ritz_diagnostics(const double* alpha, const double* beta, int32_t s, double tol, double* nodes,
                                double* weights, double* resid, int32_t* copies, int32_t* spurious,
                                int32_t* n_ghosts);

/* Per transformer layer b (section 6): out_host[3b..3b+2] = ||a_b||^2, ||b_b||^2,
 * <a_b, b_b> over the parameters of layer b; a, b float32 [P] on device. */
fdh_status fdh_block_stats(fdh_ctx* ctx, const float* a_dev, const float* b_dev, double* out_host);

/* fdh_block_stats for callers that cannot allocate device memory (code under
 * stream capture, tight serving loops, harnesses that forbid allocation): the
 * same statistics and the same kernels, with the partial sums in a fixed
 * 16 KiB device array that the library holds on every GPU it runs on until
 * the process ends, instead of the workspace.  Needs no workspace and calls
 * no device allocator.  At most 256 transformer layers (FDH_ERR_UNSUPPORTED
 * beyond, before any launch).  All calls on one GPU share that array: calls
 * that overlap on one GPU (other host threads or streams) race and must be
 * serialised by the caller.  Waits for the context stream. */
fdh_status fdh_block_stats_noalloc(fdh_ctx* ctx, const float* a_dev, const float* b_dev, double* out_host);

/* Block-diagonal hypothesis test (section 6, Exp I) on the bound operator:
 * h = H v, and for every transformer layer b, h_b = H v^(b) where v^(b) is v
 * with all entries outside layer b set to zero (not renormalised).  For each b,
 * stats_host[4b + 0] = ||h^(b) - h_b^(b)||, [4b + 1] = that over ||h^(b)||,
 * [4b + 2] = cosine of h^(b) and h_b^(b), [4b + 3] = ||h^(b)||, all restricted
 * to the parameters of layer b.  Runs L + 1 FD-HVPs; v: float32 [P] on device.
 * Needs a bound operator and a workspace planned with m >= 1 (its Lanczos vectors are
 * used as scratch).  Waits for the stream. */
fdh_status fdh_block_diagonal(fdh_ctx* ctx, const float* v_dev, double* stats_host);

/* Conjugate gradient for the damped inverse HVP on the bound operator: solves
 * (H + lambda I) x = b from x_0 = 0 (CG-based inverse-HVP solvers are the
 * second consumer the introduction and section 4 name; the method is that of
 * Hestenes and Stiefel).  b_dev, x_dev: float32 [P] on device, x overwritten,
 * not aliasing b.  Stops after max_iters steps or once ||r_k|| <= rel_tol ||b||;
 * res_host[max_iters + 1] receives ||r_0|| = ||b||, ||r_1||, ..., ||r_s||
 * (s = *steps_done, zeros after).  Returns FDH_BREAKDOWN, with x = x_s, when a
 * direction of non-positive curvature ((p, (H + lambda I) p) <= 0) stops it:
 * raise lambda.  Each step is one FD-HVP plus three vector passes; fp32
 * vectors, fp64 scalars with deterministic reductions; two scalars are read
 * back per step (the call waits for the stream).  Needs a bound operator and a
 * workspace planned with m >= 1 (its Lanczos vectors hold r, p and A p). */
fdh_status fdh_cg_solve(fdh_ctx* ctx, const float* b_dev, double lambda, int32_t max_iters, double rel_tol,
                        float* x_dev, double* res_host, int32_t* steps_done);

/* Number of transformer layers (blocks for fdh_block_stats). */
int32_t fdh_num_blocks(const fdh_ctx* ctx);

/* Message for the most recent error on this context (never NULL). */
const char* fdh_last_error(const fdh_ctx* ctx);

#ifdef __cplusplus
}
#endif
#endif /* FDHVP_H */
