// Host-side engine: parameter layout, workspace plan, the lockstep HVP and the
// Lanczos / SLQ drivers.
#pragma once
#include <string>
#include <vector>

#include "../../include/fdhvp.h"
#include "kernels.h"

namespace fdh {

struct ParamRef {
  int64_t off = -1;
  int64_t rows = 0, cols = 0;
  bool valid() const { return off >= 0; }
};

struct LayerRefs {
  ParamRef n1g, n1b, wqkv, bqkv, wo, bo, n2g, n2b, w1, b1, w2, b2;
};

struct Entry {
  std::string name;
  int64_t off, numel, rows, cols;
  int layer, kind;
};

struct BatchRef {  // one token batch of a bound dataset (device pointers, caller-owned)
  const int32_t* tok = nullptr;
  const int32_t* lab = nullptr;  // nullptr: next-token targets
  int B = 0, S = 0;
};

struct Span {  // carve of the workspace
  size_t off = 0, bytes = 0;
};

// Optional per-launch timing with HIP events on the context stream (testing
// hook used by the benchmark).  Categories: 0 GEMM, 1 Lanczos vector kernels,
// 2 fused attention (forward launch, backward launches).
struct Timing {
  static constexpr int NCAT = 4;
  static constexpr size_t POOL = 8192;
  bool on = false;
  std::vector<hipEvent_t> ev;
  size_t used = 0;
  struct Rec { int cat, e0; double flops, bytes; };
  std::vector<Rec> recs;
  double ms[NCAT] = {}, flops[NCAT] = {}, bytes[NCAT] = {};
  double count[NCAT] = {};
  hipError_t begin(hipStream_t s, int* e0);
  hipError_t end(hipStream_t s, int cat, int e0, double fl, double by);
  hipError_t harvest(hipStream_t s);
  void reset() { for (int i = 0; i < NCAT; ++i) ms[i] = flops[i] = bytes[i] = count[i] = 0.0; }
  ~Timing();
};

int ritz_diagnostics(const double* alpha, const double* beta, int s, double tol, double* nodes, double* weights,
                     double* resid, int32_t* copies, int32_t* spurious, int32_t* ghosts);

// One carve of the workspace: the span of every buffer for a plan (largest
// token batch, Lanczos steps and options) and the attention path it serves.
// Engine::plan fills a WsLayout; the engine adopts it only once a workspace
// large enough for it has been handed over, so that size queries never move
// the buffers in use.
struct WsLayout {
  struct LayerSpans {
    Span x_in_m, x_in_d, a_m, a_d, qkv_m, qkv_d, P_m, P_d, st, o_m, o_d, xmid_m, xmid_d, b_m, b_d, u_m, u_d, z_m, z_d;
  };
  std::vector<LayerSpans> ls;
  Span xL_m, xL_d, f_m, f_d, lo, sc_m, sc_d, log_m, log_d, dlog_m, dlog_d, rowloss, losses;
  Span dx0_m, dx0_d, dx1_m, dx1_d, dxo_m, dxo_d, dz_m, dz_d, dgu_m, dgu_d, dudf, db_m, db_d, gpart, do_m, do_d, dS_m, dS_d;
  Span dqkv_m, dqkv_d, dqkvo_m, dqkvo_d, gqa_m, gqa_d, dl, da_m, da_d, colpart, keys, rope, cdf, gpartial, bpart, bout;
  Span tcount;  // two int64 counters of fdh_bind_dataset
  Span nfflag;  // non-finite flags of the input direction and the product (two int32)
  Span wsplit;  // split-K partial products of the weight-gradient GEMMs
  Span lz_w, lz_q, lz_qp, lz_basis, lz_alpha, lz_beta, lz_coef, lz_gram, lz_partial, lz_flag, lz_maxabs;
  int64_t lz_ldq = 0;   // basis row stride (elements, multiple of 8)
  int lz_dev_rows = 0;  // basis rows held in the workspace
  // attention path: fused kernels (bf16, head dim 64 or 128, S a multiple of
  // 128) or score/probability matrices in the workspace
  bool fused = false;
  // activation recomputation: only each layer's input pair x_in is kept; the
  // other spans of every layer alias one shared set, which the backward refills
  // by running that layer's forward again (x_in -> z) just before its backward
  bool rc = false;
  int planB = 0, planS = 0, planM = 0;
  fdh_lanczos_opts planO{};
  size_t total = 0;     // bytes the carve needs
};

class Engine : public WsLayout {
 public:
  explicit Engine(const fdh_model_config& cfg, hipStream_t stream);

  // configuration
  fdh_model_config cfg;
  hipStream_t stream;
  bool gpt2 = false, llama = false, quad = false, bf16 = false;
  int L = 0, d = 0, Hq = 0, Hk = 0, dh = 0, F = 0, V = 0, Smax = 0, qkvd = 0;
  int64_t P = 0;
  std::vector<Entry> entries;
  std::vector<LayerRefs> layers;
  ParamRef wte, wpe, head, nfg, nfb;
  std::string err;

  // workspace
  char* ws = nullptr;
  size_t ws_bytes = 0;
  bool force_unfused = false;   // testing: plan the unfused path even where the fused one applies
  bool force_unsplit = false;   // testing: weight-gradient GEMMs over the whole token range
  bool force_unpaired = false;  // testing: no weight-gradient GEMMs paired in one launch
  bool recompute = false;       // plan (and run) with activation recomputation
  // the carve for token batches up to [B, S] and m Lanczos steps with options
  // o (o may be null when m == 0), written into *out; changes nothing else
  size_t plan(int B, int S, int m, const fdh_lanczos_opts* o, WsLayout* out) const;
  // plan, check that bytes covers it, then adopt the carve and the buffer
  int set_workspace(void* dev, size_t bytes, int B, int S, int m, const fdh_lanczos_opts* o);
  // order-sensitive digest of the adopted carve (testing)
  uint64_t layout_digest() const;

  // operator binding for Lanczos / CG / the block-diagonal test: parameters,
  // step and the batches whose token-weighted average the operator is
  std::vector<BatchRef> b_data;
  const void* b_params = nullptr;
  double b_eps = 0.0;
  double b_inv_n = 0.0;   // scale of every kept cross-entropy row (1 / targets, or 1 for a sum)
  int64_t b_targets = 0;
  bool bound = false;
  const float* quad_diag = nullptr;
  Timing timing;

  // entry points (return fdh_status)
  int hvp(const void* params, const float* v, double eps, const int32_t* tok, int B, int S, float* hv);
  int hvp_batches(const void* params, const float* v, double eps, const BatchRef* bt, int nb, double inv_n, float* hv);
  int bind_batches(const void* params, const BatchRef* bt, int nb, double eps, int reduction, int64_t* targets);
  int hvp_bound(const float* v, float* hv);        // checked: waits, reports NaN/Inf and bad tokens
  int hvp_bound_async(const float* v, float* hv);  // enqueued only (Lanczos, CG, block test)
  int last_losses(double* lp, double* lm);
  int lanczos(int m, uint64_t seed, const fdh_lanczos_opts& o, double* alpha, double* beta, int* steps);
  int slq(int probes, int m, uint64_t seed, const fdh_lanczos_opts& o, double* nodes, double* weights, int* steps,
          double* trace);
  int init_params(void* params, uint64_t seed);
  int make_tokens(int32_t* tok, int B, int S, uint64_t seed, int dist);
  int random_vector(float* out, uint64_t seed, int kind);
  int block_stats(const float* a, const float* b, double* out);
  int block_diagonal(const float* v, double* out);
  int cg_solve(const float* b, double lam, int max_iters, double rel_tol, float* x, double* res, int* steps);
  int set_basis_offload(int device_rows, void* host, size_t bytes);
  std::vector<int64_t> layer_ranges() const;

 private:
  int check_batch(const int32_t* tok, int B, int S);
  int finish_checked(const float* hv);
  template <typename T>
  int hvp_t(const T* th, const float* v, double eps, const int32_t* tok, const int32_t* lab, int B, int S, double inv_n,
            bool acc, float* hv);
  template <typename B> int lanczos_t(int m, uint64_t seed, const fdh_lanczos_opts& o, double* alpha, double* beta, int* steps);
  template <typename T> void* wsp(const Span& s) const { return (void*)(ws + s.off); }

  // basis offload: at most off_rows rows in the workspace (-1: all), the rest
  // in caller-owned pinned host memory (device-side address)
  int off_rows = -1;
  void* host_rows_dev = nullptr;
  size_t host_rows_bytes = 0;
  // set by the Lanczos normalisation when it already wrote lo = eps * v for
  // the next HVP (of this v and eps); consumed by that HVP
  const float* lo_for_v = nullptr;
  double lo_for_eps = 0.0;
};

}  // namespace fdh
