// C ABI (include/fdhvp.h): argument validation and dispatch to the engine.
// No exception crosses this boundary.
#include <cstring>
#include <mutex>
#include <new>
#include <string>

#include "engine.h"

struct fdh_ctx {
  fdh::Engine* eng = nullptr;
  std::string err;
};

namespace {

fdh_status guard(fdh_ctx* c, int rc) {
  if (rc < 0 && c && c->eng) c->err = c->eng->err;
  return (fdh_status)rc;
}

template <typename F>
fdh_status run(fdh_ctx* c, F&& f) {
  if (!c || !c->eng) return FDH_ERR_INVALID_ARG;
  try {
    return guard(c, f(*c->eng));
  } catch (const std::bad_alloc&) {
    c->err = "host allocation failed";
    return FDH_ERR_INVALID_ARG;
  } catch (...) {
    c->err = "unexpected host exception";
    return FDH_ERR_INVALID_ARG;
  }
}

const char* validate(const fdh_model_config* cfg) {
  if (!cfg) return "null config";
  if (cfg->dtype != FDH_F32 && cfg->dtype != FDH_BF16) return "dtype must be FDH_F32 or FDH_BF16";
  if (cfg->family == FDH_FAMILY_QUAD_DIAG) return cfg->quad_n > 0 ? nullptr : "quad_n must be positive";
  if (cfg->family != FDH_FAMILY_GPT2 && cfg->family != FDH_FAMILY_LLAMA) return "unknown family";
  if (cfg->n_layers < 0 || cfg->d_model < 1 || cfg->n_heads < 1 || cfg->n_kv_heads < 1 || cfg->d_ff < 1 ||
      cfg->vocab < 2 || cfg->max_seq < 2)
    return "non-positive model size";
  if (cfg->d_model % cfg->n_heads) return "n_heads must divide d_model";
  if (cfg->n_heads % cfg->n_kv_heads) return "n_kv_heads must divide n_heads";
  if (cfg->family == FDH_FAMILY_GPT2 && cfg->n_kv_heads != cfg->n_heads) return "GPT-2 family has n_kv_heads == n_heads";
  const int dh = cfg->d_model / cfg->n_heads;
  if (dh % 8 || cfg->d_model % 8 || cfg->d_ff % 8 || cfg->vocab % 8) return "d_model, head_dim, d_ff, vocab must be multiples of 8";
  if (cfg->vocab >= (1 << 18)) return "vocab must be < 2^18";
  if (!(cfg->norm_eps > 0.f)) return "norm_eps must be positive";
  if (cfg->family == FDH_FAMILY_LLAMA && !(cfg->rope_base > 1.f)) return "rope_base must be > 1";
  return nullptr;
}

}  // namespace

extern "C" {

int32_t fdh_api_version(void) { return FDH_API_VERSION; }

fdh_status fdh_create(const fdh_model_config* cfg, void* hip_stream, fdh_ctx** out) {
  if (!out) return FDH_ERR_INVALID_ARG;
  *out = nullptr;
  if (validate(cfg)) return FDH_ERR_INVALID_ARG;
  fdh_ctx* c = new (std::nothrow) fdh_ctx;
  if (!c) return FDH_ERR_INVALID_ARG;
  try {
    c->eng = new fdh::Engine(*cfg, (hipStream_t)hip_stream);
  } catch (...) {
    delete c;
    return FDH_ERR_INVALID_ARG;
  }
  *out = c;
  return FDH_OK;
}

void fdh_destroy(fdh_ctx* ctx) {
  if (!ctx) return;
  delete ctx->eng;
  delete ctx;
}

int64_t fdh_num_params(const fdh_ctx* ctx) { return (ctx && ctx->eng) ? ctx->eng->P : -1; }

fdh_status fdh_ritz_diagnostics(const double* alpha, const double* beta, int32_t s, double tol, double* nodes,
                                double* weights, double* resid, int32_t* copies, int32_t* spurious, int32_t* n_ghosts) {
  try {
    return (fdh_status)fdh::ritz_diagnostics(alpha, beta, s, tol, nodes, weights, resid, copies, spurious, n_ghosts);
  } catch (...) {
    return FDH_ERR_INVALID_ARG;
  }
}

int32_t fdh_num_blocks(const fdh_ctx* ctx) { return (ctx && ctx->eng) ? ctx->eng->L : -1; }

fdh_status fdh_param_layout(const fdh_ctx* ctx, fdh_block* out, int32_t cap, int32_t* n) {
  if (!ctx || !ctx->eng || !n || cap < 0 || (cap > 0 && !out)) return FDH_ERR_INVALID_ARG;
  const auto& E = ctx->eng->entries;
  *n = (int32_t)E.size();
  for (int32_t i = 0; i < cap && i < (int32_t)E.size(); ++i) {
    std::memset(&out[i], 0, sizeof(fdh_block));
    std::strncpy(out[i].name, E[i].name.c_str(), sizeof(out[i].name) - 1);
    out[i].offset = E[i].off;
    out[i].numel = E[i].numel;
    out[i].rows = E[i].rows;
    out[i].cols = E[i].cols;
    out[i].layer = E[i].layer;
    out[i].kind = E[i].kind;
  }
  return FDH_OK;
}

fdh_status fdh_workspace_bytes(const fdh_ctx* ctx, int32_t B, int32_t S, int32_t m, const fdh_lanczos_opts* o,
                               size_t* bytes) {
  if (!ctx || !ctx->eng || !bytes || B < 0 || S < 0 || m < 0 || (m > 0 && !o)) return FDH_ERR_INVALID_ARG;
  try {
    *bytes = ctx->eng->plan(B, S, m, o, nullptr);  // a query: the adopted carve is left alone
  } catch (...) {
    return FDH_ERR_INVALID_ARG;
  }
  return FDH_OK;
}

fdh_status fdh_set_workspace(fdh_ctx* ctx, void* dev, size_t bytes, int32_t B, int32_t S, int32_t m,
                             const fdh_lanczos_opts* o) {
  return run(ctx, [&](fdh::Engine& e) { return e.set_workspace(dev, bytes, B, S, m, o); });
}

fdh_status fdh_set_recompute(fdh_ctx* ctx, int32_t on) {
  return run(ctx, [&](fdh::Engine& e) -> int {
    e.recompute = on != 0;
    return FDH_OK;
  });
}

fdh_status fdh_init_params(fdh_ctx* ctx, void* params_dev, uint64_t seed) {
  return run(ctx, [&](fdh::Engine& e) { return e.init_params(params_dev, seed); });
}

fdh_status fdh_make_tokens(fdh_ctx* ctx, int32_t* tokens_dev, int32_t B, int32_t S, uint64_t seed, int32_t dist) {
  return run(ctx, [&](fdh::Engine& e) { return e.make_tokens(tokens_dev, B, S, seed, dist); });
}

fdh_status fdh_random_vector(fdh_ctx* ctx, float* out_dev, uint64_t seed, int32_t kind) {
  return run(ctx, [&](fdh::Engine& e) { return e.random_vector(out_dev, seed, kind); });
}

fdh_status fdh_set_quad_diag(fdh_ctx* ctx, const float* diag_dev) {
  return run(ctx, [&](fdh::Engine& e) -> int {
    if (!e.quad) { e.err = "not a QUAD_DIAG context"; return FDH_ERR_STATE; }
    if (!diag_dev) { e.err = "null diagonal"; return FDH_ERR_INVALID_ARG; }
    e.quad_diag = diag_dev;
    return FDH_OK;
  });
}

fdh_status fdh_hvp(fdh_ctx* ctx, const void* params_dev, const float* v_dev, double eps, const int32_t* tokens_dev,
                   int32_t B, int32_t S, float* hv_dev) {
  return run(ctx, [&](fdh::Engine& e) { return e.hvp(params_dev, v_dev, eps, tokens_dev, B, S, hv_dev); });
}

fdh_status fdh_last_losses(fdh_ctx* ctx, double* loss_plus, double* loss_minus) {
  return run(ctx, [&](fdh::Engine& e) { return e.last_losses(loss_plus, loss_minus); });
}

fdh_status fdh_bind(fdh_ctx* ctx, const void* params_dev, const int32_t* tokens_dev, int32_t B, int32_t S, double eps) {
  return run(ctx, [&](fdh::Engine& e) -> int {
    if (e.quad) return e.bind_batches(params_dev, nullptr, 0, eps, FDH_REDUCE_MEAN, nullptr);
    fdh::BatchRef b;
    b.tok = tokens_dev;
    b.B = B;
    b.S = S;
    return e.bind_batches(params_dev, &b, 1, eps, FDH_REDUCE_MEAN, nullptr);
  });
}

fdh_status fdh_bind_dataset(fdh_ctx* ctx, const void* params_dev, const fdh_batch* batches, int32_t nbatch, double eps,
                            int32_t reduction, int64_t* n_targets) {
  return run(ctx, [&](fdh::Engine& e) -> int {
    if (nbatch < 0 || (nbatch > 0 && !batches)) { e.err = "bad batch list"; return FDH_ERR_INVALID_ARG; }
    std::vector<fdh::BatchRef> bt((size_t)nbatch);
    for (int i = 0; i < nbatch; ++i) {
      bt[i].tok = batches[i].tokens;
      bt[i].lab = batches[i].labels;
      bt[i].B = batches[i].B;
      bt[i].S = batches[i].S;
    }
    return e.bind_batches(params_dev, bt.data(), nbatch, eps, reduction, n_targets);
  });
}

fdh_status fdh_set_basis_offload(fdh_ctx* ctx, int32_t device_rows, void* host_rows, size_t host_bytes) {
  return run(ctx, [&](fdh::Engine& e) { return e.set_basis_offload(device_rows, host_rows, host_bytes); });
}

fdh_status fdh_hvp_bound(fdh_ctx* ctx, const float* v_dev, float* hv_dev) {
  return run(ctx, [&](fdh::Engine& e) { return e.hvp_bound(v_dev, hv_dev); });
}

fdh_status fdh_lanczos(fdh_ctx* ctx, int32_t m, uint64_t probe_seed, const fdh_lanczos_opts* o, double* alpha_host,
                       double* beta_host, int32_t* steps_done) {
  return run(ctx, [&](fdh::Engine& e) -> int {
    if (!o) { e.err = "null options"; return FDH_ERR_INVALID_ARG; }
    int s = 0;
    int rc = e.lanczos(m, probe_seed, *o, alpha_host, beta_host, &s);
    if (steps_done) *steps_done = s;
    return rc;
  });
}

fdh_status fdh_slq_density(fdh_ctx* ctx, int32_t probes, int32_t m, uint64_t seed, const fdh_lanczos_opts* o,
                           double* nodes_host, double* weights_host, int32_t* steps_done, double* trace_est) {
  return run(ctx, [&](fdh::Engine& e) -> int {
    if (!o) { e.err = "null options"; return FDH_ERR_INVALID_ARG; }
    return e.slq(probes, m, seed, *o, nodes_host, weights_host, steps_done, trace_est);
  });
}

fdh_status fdh_block_stats(fdh_ctx* ctx, const float* a_dev, const float* b_dev, double* out_host) {
  return run(ctx, [&](fdh::Engine& e) { return e.block_stats(a_dev, b_dev, out_host); });
}

}  // extern "C"

// ---- allocation-free block statistics --------------------------------------
// The partial sums of fdh_block_stats_noalloc live in one file-scope device
// array per GPU instead of the workspace: 256 workgroup partials of four sums,
// then four sums per block, for at most NOALLOC_MAX_BLOCKS blocks (16 KiB).
// Host code never passes the array's name to a kernel (on the host it only
// stands in for the symbol): its device address is looked up once per device
// with hipGetSymbolAddress and that address is used everywhere.
constexpr int NOALLOC_MAX_BLOCKS = 256;
constexpr int NOALLOC_PARTIALS = 256 * 4;  // launch_block_stats: 256 workgroups x 4 sums
static __device__ __align__(256) double scratch[NOALLOC_PARTIALS + 4 * NOALLOC_MAX_BLOCKS];

namespace {
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
double* g_scratch_ptr[MAX_DEVICES] = {};

// device address of this device's scratch array (looked up on first use)
hipError_t scratch_ptr(double** out) {
  int dev = 0;
  hipError_t r = hipGetDevice(&dev);
  if (r != hipSuccess) return r;
  if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    r = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (r != hipSuccess) return r;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = (double*)p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}
}  // namespace

extern "C" {

fdh_status fdh_block_stats_noalloc(fdh_ctx* ctx, const float* a_dev, const float* b_dev, double* out_host) {
  return run(ctx, [&](fdh::Engine& e) -> int {
    if (e.quad || !a_dev || !b_dev || !out_host) { e.err = "bad block_stats arguments"; return FDH_ERR_INVALID_ARG; }
    if (e.L > NOALLOC_MAX_BLOCKS) {
      e.err = "fdh_block_stats_noalloc handles at most 256 blocks; use fdh_block_stats";
      return FDH_ERR_UNSUPPORTED;
    }
    double* sp = nullptr;
    hipError_t r = scratch_ptr(&sp);
    if (r != hipSuccess) { e.err = std::string("scratch symbol: ") + hipGetErrorString(r); return FDH_ERR_HIP; }
    double* part = sp;
    double* sums = sp + NOALLOC_PARTIALS;
    // layer ranges straight from the layout (per-layer entries are contiguous)
    for (int l = 0; l < e.L; ++l) {
      int64_t rg[2] = {-1, -1};
      for (const fdh::Entry& en : e.entries)
        if (en.layer == l) {
          if (rg[0] < 0) rg[0] = en.off;
          rg[1] = en.off + en.numel;
        }
      r = fdh::launch_block_stats(a_dev, b_dev, rg, 1, part, sums + 4 * l, e.stream);
      if (r != hipSuccess) { e.err = std::string("block stats launch: ") + hipGetErrorString(r); return FDH_ERR_HIP; }
    }
    double h[4 * NOALLOC_MAX_BLOCKS];
    if (e.L > 0) {
      r = hipMemcpyAsync(h, sums, sizeof(double) * 4 * e.L, hipMemcpyDeviceToHost, e.stream);
      if (r == hipSuccess) r = hipStreamSynchronize(e.stream);
      if (r != hipSuccess) { e.err = std::string("block stats read-back: ") + hipGetErrorString(r); return FDH_ERR_HIP; }
    }
    for (int l = 0; l < e.L; ++l)
      for (int c = 0; c < 3; ++c) out_host[3 * l + c] = h[4 * l + c];
    return FDH_OK;
  });
}

fdh_status fdh_block_diagonal(fdh_ctx* ctx, const float* v_dev, double* stats_host) {
  return run(ctx, [&](fdh::Engine& e) { return e.block_diagonal(v_dev, stats_host); });
}

fdh_status fdh_cg_solve(fdh_ctx* ctx, const float* b_dev, double lambda, int32_t max_iters, double rel_tol,
                        float* x_dev, double* res_host, int32_t* steps_done) {
  return run(ctx, [&](fdh::Engine& e) -> int {
    int s = 0;
    int rc = e.cg_solve(b_dev, lambda, max_iters, rel_tol, x_dev, res_host, &s);
    if (steps_done) *steps_done = s;
    return rc;
  });
}

const char* fdh_last_error(const fdh_ctx* ctx) {
  if (!ctx) return "null context";
  return ctx->err.c_str();
}

}  // extern "C"

// ---- testing hooks (include/fdhvp_testing.h) ----
#include "../../include/fdhvp_testing.h"

extern "C" fdh_status fdh_testing_gemm(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t batch, int32_t a_kmajor,
                                       int32_t b_kmajor, const void* A, const void* B, const void* A2, const void* B2,
                                       float* C, int32_t causal, float alpha, int32_t tile, void* hip_stream) {
  if (!A || !B || !C || (!A2) != (!B2) || M < 0 || N < 0 || K < 0 || batch < 1 || causal < 0 || causal > 3 ||
      tile < 0 || tile > 8)
    return FDH_ERR_INVALID_ARG;
  fdh::GemmArgs g;
  g.tile = tile;
  g.M = M; g.N = N; g.K = K; g.nbatch = batch; g.inner_count = 1;
  g.npairs = A2 ? 2 : 1;
  const void* As[2] = {A, A2};
  const void* Bs[2] = {B, B2};
  for (int p = 0; p < g.npairs; ++p) {
    g.A[p].ptr = As[p];
    g.A[p].s_row = a_kmajor ? K : 1;
    g.A[p].s_k = a_kmajor ? 1 : M;
    g.A[p].s_outer = (int64_t)M * K;
    g.B[p].ptr = Bs[p];
    g.B[p].s_row = b_kmajor ? K : 1;
    g.B[p].s_k = b_kmajor ? 1 : N;
    g.B[p].s_outer = (int64_t)N * K;
  }
  g.C = C; g.ldc = N; g.c_outer = (int64_t)M * N;
  g.alpha = alpha;
  g.causal = causal;
  hipError_t r;
  if (dtype == FDH_BF16) {
    if (fdh::gemm_check<fdh::bf16_t>(g)) return FDH_ERR_UNSUPPORTED;
    r = fdh::gemm<fdh::bf16_t>(g, (hipStream_t)hip_stream);
  } else if (dtype == FDH_F32) {
    if (fdh::gemm_check<float>(g)) return FDH_ERR_UNSUPPORTED;
    r = fdh::gemm<float>(g, (hipStream_t)hip_stream);
  } else {
    return FDH_ERR_INVALID_ARG;
  }
  return r == hipSuccess ? FDH_OK : FDH_ERR_HIP;
}

extern "C" fdh_status fdh_testing_gemm_pair(int32_t M0, int32_t N0, int32_t K0, int32_t batch0, int32_t M1,
                                            int32_t N1, int32_t K1, int32_t batch1, int32_t a_kmajor,
                                            int32_t b_kmajor, const void* A0, const void* B0, const void* A20,
                                            const void* B20, float* C0, const void* A1, const void* B1,
                                            const void* A21, const void* B21, float* C1, float alpha, int32_t tile,
                                            void* hip_stream) {
  if (!A0 || !B0 || !C0 || !A1 || !B1 || !C1 || (!A20) != (!B20) || (!A21) != (!B21) || M0 < 0 || N0 < 0 ||
      K0 < 0 || M1 < 0 || N1 < 0 || K1 < 0 || batch0 < 1 || batch1 < 1 || (tile != 6 && tile != 8))
    return FDH_ERR_INVALID_ARG;
  fdh::GemmArgs g[2];
  const int32_t Ms[2] = {M0, M1}, Ns[2] = {N0, N1}, Ks[2] = {K0, K1}, Bs_[2] = {batch0, batch1};
  const void* As[2][2] = {{A0, A20}, {A1, A21}};
  const void* Bs[2][2] = {{B0, B20}, {B1, B21}};
  float* Cs[2] = {C0, C1};
  for (int q = 0; q < 2; ++q) {
    fdh::GemmArgs& a = g[q];
    a.tile = tile;
    a.M = Ms[q]; a.N = Ns[q]; a.K = Ks[q];
    a.nbatch = Bs_[q]; a.inner_count = 1;
    a.npairs = As[q][1] ? 2 : 1;
    for (int p = 0; p < a.npairs; ++p) {
      a.A[p].ptr = As[q][p];
      a.A[p].s_row = a_kmajor ? Ks[q] : 1;
      a.A[p].s_k = a_kmajor ? 1 : Ms[q];
      a.A[p].s_outer = (int64_t)Ms[q] * Ks[q];
      a.B[p].ptr = Bs[q][p];
      a.B[p].s_row = b_kmajor ? Ks[q] : 1;
      a.B[p].s_k = b_kmajor ? 1 : Ns[q];
      a.B[p].s_outer = (int64_t)Ns[q] * Ks[q];
    }
    a.C = Cs[q]; a.ldc = Ns[q]; a.c_outer = (int64_t)Ms[q] * Ns[q];
    a.alpha = alpha;
    if (a.M < 8 || a.N < 8 || fdh::gemm_check<fdh::bf16_t>(a)) return FDH_ERR_UNSUPPORTED;
  }
  const hipError_t r = fdh::gemm_pair<fdh::bf16_t>(g[0], g[1], (hipStream_t)hip_stream);
  return r == hipSuccess ? FDH_OK : FDH_ERR_HIP;
}

extern "C" fdh_status fdh_testing_unfused_attention(fdh_ctx* ctx, int32_t on) {
  return run(ctx, [&](fdh::Engine& e) -> int {
    e.force_unfused = on != 0;
    return FDH_OK;
  });
}

extern "C" fdh_status fdh_testing_unsplit_wgrad(fdh_ctx* ctx, int32_t on) {
  return run(ctx, [&](fdh::Engine& e) -> int {
    if (on < 0 || on > 2) {
      e.err = "unsplit_wgrad: mode must be 0, 1 or 2";
      return FDH_ERR_INVALID_ARG;
    }
    e.force_unsplit = on == 1;
    e.force_unpaired = on != 0;
    return FDH_OK;
  });
}

extern "C" fdh_status fdh_testing_timing(fdh_ctx* ctx, int32_t enable) {
  return run(ctx, [&](fdh::Engine& e) -> int {
    if (e.timing.on) {
      hipError_t r = e.timing.harvest(e.stream);
      if (r != hipSuccess) { e.err = "timing harvest"; return FDH_ERR_HIP; }
    }
    e.timing.on = enable != 0;
    e.timing.reset();
    return FDH_OK;
  });
}

extern "C" fdh_status fdh_testing_timing_read(fdh_ctx* ctx, double* out16) {
  return run(ctx, [&](fdh::Engine& e) -> int {
    if (!out16) { e.err = "null output"; return FDH_ERR_INVALID_ARG; }
    hipError_t r = e.timing.harvest(e.stream);
    if (r != hipSuccess) { e.err = "timing harvest"; return FDH_ERR_HIP; }
    for (int c = 0; c < fdh::Timing::NCAT; ++c) {
      out16[4 * c + 0] = e.timing.count[c];
      out16[4 * c + 1] = e.timing.ms[c];
      out16[4 * c + 2] = e.timing.flops[c];
      out16[4 * c + 3] = e.timing.bytes[c];
    }
    e.timing.reset();
    return FDH_OK;
  });
}

extern "C" fdh_status fdh_testing_layout_digest(const fdh_ctx* ctx, uint64_t* out) {
  if (!ctx || !ctx->eng || !out) return FDH_ERR_INVALID_ARG;
  *out = ctx->eng->layout_digest();
  return FDH_OK;
}

extern "C" fdh_status fdh_testing_copy(void* dst, const void* src, size_t bytes, void* hip_stream) {
  if (!dst || !src || (bytes & 15) || (reinterpret_cast<uintptr_t>(dst) & 15) || (reinterpret_cast<uintptr_t>(src) & 15))
    return FDH_ERR_INVALID_ARG;
  return fdh::launch_copy16(dst, src, bytes, (hipStream_t)hip_stream) == hipSuccess ? FDH_OK : FDH_ERR_HIP;
}
