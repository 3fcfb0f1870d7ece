// Host engine: layout, workspace plan, lockstep FD-HVP, Lanczos and SLQ.
//
// The FD-HVP (section 3.1, Eq. grad-fd-hvp; Algorithm 1 with one batch) needs
// the gradients at theta + eps v and theta - eps v.  Both gradient passes run
// at once: every activation and every upstream gradient is held as its mean m
// and half difference d over the two points.  A linear layer y = x W^T with
// W = theta +- eps v then splits exactly into
//     y.m = x.m theta^T                      (+ x.d (eps v)^T, O(eps^2), below the rounding of y.m: not formed)
//     y.d = x.d theta^T + x.m (eps v)^T
// and the weight gradient needs only its half difference
//     (g+ - g-)/2 = dy.m^T x.d + dy.d^T x.m,   so   Hv_W = (dy.m^T x.d + dy.d^T x.m) / eps.
// Every non-linear step (norms, softmax, GELU/SwiGLU, cross-entropy) is
// evaluated at both points in fp64 inside its kernel.  theta is never written.
#include "engine.h"

#include <algorithm>
#include <functional>
#include <queue>
#include <vector>
#include <type_traits>
#include <cmath>
#include <cstring>

namespace fdh {

#define CK(x)                                                                     \
  do {                                                                            \
    hipError_t e_ = (x);                                                          \
    if (e_ != hipSuccess) {                                                       \
      err = std::string(#x) + ": " + hipGetErrorString(e_);                       \
      return FDH_ERR_HIP;                                                         \
    }                                                                             \
  } while (0)

namespace {

GemmOperand kmaj(const void* p, int64_t ld) {
  GemmOperand o;
  o.ptr = p;
  o.s_row = ld;
  o.s_k = 1;
  return o;
}
GemmOperand mnmaj(const void* p, int64_t ld) {
  GemmOperand o;
  o.ptr = p;
  o.s_row = 1;
  o.s_k = ld;
  return o;
}

constexpr size_t ALIGN = 256;

}  // namespace

Engine::Engine(const fdh_model_config& c, hipStream_t s) : cfg(c), stream(s) {
  quad = cfg.family == FDH_FAMILY_QUAD_DIAG;
  gpt2 = cfg.family == FDH_FAMILY_GPT2;
  llama = cfg.family == FDH_FAMILY_LLAMA;
  bf16 = cfg.dtype == FDH_BF16;
  if (quad) {
    P = cfg.quad_n;
    entries.push_back({"theta", 0, P, P, 1, -1, FDH_PARAM_MATRIX});
    return;
  }
  L = cfg.n_layers;
  d = cfg.d_model;
  Hq = cfg.n_heads;
  Hk = cfg.n_kv_heads;
  dh = d / Hq;
  F = cfg.d_ff;
  V = cfg.vocab;
  Smax = cfg.max_seq;
  qkvd = (Hq + 2 * Hk) * dh;
  int64_t off = 0;
  auto add = [&](const std::string& name, int64_t rows, int64_t cols, int layer, int kind) {
    ParamRef r;
    r.off = off;
    r.rows = rows;
    r.cols = cols;
    entries.push_back({name, off, rows * cols, rows, cols, layer, kind});
    off += rows * cols;
    return r;
  };
  layers.resize(L);
  if (gpt2) {
    wte = add("wte", V, d, -1, FDH_PARAM_MATRIX);
    wpe = add("wpe", Smax, d, -1, FDH_PARAM_MATRIX);
    for (int l = 0; l < L; ++l) {
      const std::string p = "h" + std::to_string(l) + ".";
      LayerRefs& R = layers[l];
      R.n1g = add(p + "ln1.g", d, 1, l, FDH_PARAM_GAIN);
      R.n1b = add(p + "ln1.b", d, 1, l, FDH_PARAM_BIAS);
      R.wqkv = add(p + "wqkv", 3 * d, d, l, FDH_PARAM_MATRIX);
      R.bqkv = add(p + "bqkv", 3 * d, 1, l, FDH_PARAM_BIAS);
      R.wo = add(p + "wo", d, d, l, FDH_PARAM_MATRIX);
      R.bo = add(p + "bo", d, 1, l, FDH_PARAM_BIAS);
      R.n2g = add(p + "ln2.g", d, 1, l, FDH_PARAM_GAIN);
      R.n2b = add(p + "ln2.b", d, 1, l, FDH_PARAM_BIAS);
      R.w1 = add(p + "w1", F, d, l, FDH_PARAM_MATRIX);
      R.b1 = add(p + "b1", F, 1, l, FDH_PARAM_BIAS);
      R.w2 = add(p + "w2", d, F, l, FDH_PARAM_MATRIX);
      R.b2 = add(p + "b2", d, 1, l, FDH_PARAM_BIAS);
    }
    nfg = add("lnf.g", d, 1, -1, FDH_PARAM_GAIN);
    nfb = add("lnf.b", d, 1, -1, FDH_PARAM_BIAS);
    head = wte;
  } else {
    wte = add("embed", V, d, -1, FDH_PARAM_MATRIX);
    for (int l = 0; l < L; ++l) {
      const std::string p = "h" + std::to_string(l) + ".";
      LayerRefs& R = layers[l];
      R.n1g = add(p + "norm1.g", d, 1, l, FDH_PARAM_GAIN);
      R.wqkv = add(p + "wqkv", qkvd, d, l, FDH_PARAM_MATRIX);
      R.wo = add(p + "wo", d, Hq * dh, l, FDH_PARAM_MATRIX);
      R.n2g = add(p + "norm2.g", d, 1, l, FDH_PARAM_GAIN);
      R.w1 = add(p + "wgu", 2 * F, d, l, FDH_PARAM_MATRIX);
      R.w2 = add(p + "wd", d, F, l, FDH_PARAM_MATRIX);
    }
    nfg = add("normf.g", d, 1, -1, FDH_PARAM_GAIN);
    head = add("head", V, d, -1, FDH_PARAM_MATRIX);
  }
  P = off;
}

// Number of K slices for a weight-gradient GEMM (M x N output, contraction
// over the T tokens).  A grid of fewer than 128 output tiles leaves most of
// the 256 compute units idle; slicing the token range multiplies the
// workgroups, up to one full wave of 256.  Larger grids are not sliced: there
// the extra prologues, epilogues and the summation pass cost more than the
// better balance gains (measured on the 1.3B shapes).
static int wgrad_splits(int M, int N, int T_) {
  const int64_t tiles = (int64_t)((M + 255) / 256) * ((N + 255) / 256);
  if (tiles >= 128) return 1;
  int best = 1;
  for (int s : {2, 3, 4, 6, 8})
    if (T_ % (64 * s) == 0 && T_ / s >= 1024 && tiles * s <= 256) best = s;
  return best;
}

// The weight gradient of the attention output projection (Mo x No) runs in
// the same launch as the q/k/v one (Mq x Nq) when the q/k/v grid is not cut
// along the tokens and the output projection's tiles fit into the idle part
// of its last wave of 256 tiles (the 2048-wide layer: 192 + 64 tiles).  Its
// tiles then cost no extra time, where on their own they would be cut into
// token slices and summed.
static bool pair_wgrads(int Mq, int Nq, int Mo, int No, int T_) {
  const int64_t tq = (int64_t)((Mq + 255) / 256) * ((Nq + 255) / 256);
  const int64_t to = (int64_t)((Mo + 255) / 256) * ((No + 255) / 256);
  return wgrad_splits(Mq, Nq, T_) == 1 && tq % 256 != 0 && tq % 256 + to <= 256;
}

// The MLP's two weight gradients (gate/up: Ma x Na, down: Mb x Nb) in one
// launch, the down one cut into s token slices: returns s, or 0 for two
// launches of their own.  Tiles of the same depth take one time unit (a wave
// of 256 takes one), and the dispatcher hands the next tile of the grid to the
// first free compute unit; the estimate adds the slice sums (s partial
// products written and read at about 5 TB/s, against a 256 x 256 tile of two
// operand pairs at about 4.7 TFLOP/s per compute unit).  The 2048-wide layer
// at 8192 tokens: 352 + 176 tiles take 3 units in two launches, 2.25 in one
// with the down gradient in 4 slices.
static int mlp_wgrad_split(int Ma, int Na, int Mb, int Nb, int T_) {
  const int64_t ta = (int64_t)((Ma + 255) / 256) * ((Na + 255) / 256);
  const int64_t tb = (int64_t)((Mb + 255) / 256) * ((Nb + 255) / 256);
  if (wgrad_splits(Ma, Na, T_) != 1 || wgrad_splits(Mb, Nb, T_) != 1) return 0;
  auto makespan = [&](int s) {
    std::priority_queue<double, std::vector<double>, std::greater<double>> cu;
    for (int i = 0; i < 256; ++i) cu.push(0.0);
    auto take = [&](double len) {
      const double t = cu.top();
      cu.pop();
      cu.push(t + len);
    };
    for (int64_t i = 0; i < ta; ++i) take(1.0);
    for (int64_t i = 0; i < tb * s; ++i) take(1.0 / s);
    double end = 0.0;
    while (!cu.empty()) {
      end = std::max(end, cu.top());
      cu.pop();
    }
    return end;
  };
  const double apart = (double)((ta + 255) / 256 + (tb + 255) / 256);
  double best = apart - 0.25;
  int pick = 0;
  for (int s : {1, 2, 4}) {
    if (T_ % (64 * s) != 0 || T_ / s < 1024) continue;
    const double sums = s > 1 ? (double)s * Mb * Nb * 8.0 / (2.8e5 * T_) : 0.0;
    const double t = makespan(s) + sums;
    if (t < best) {
      best = t;
      pick = s;
    }
  }
  return pick;
}

// ---------------------------------------------------------------------------
// workspace plan
// ---------------------------------------------------------------------------
size_t Engine::plan(int B, int S, int m, const fdh_lanczos_opts* o, WsLayout* out) const {
  WsLayout W;
  size_t cur = 0;
  auto take = [&](Span& s, size_t bytes) {
    s.off = cur;
    s.bytes = bytes;
    cur += (bytes + ALIGN - 1) / ALIGN * ALIGN;
  };
  const size_t ob = bf16 ? 2 : 4;
  if (!quad) {
    const size_t T_ = (size_t)B * S;
    const size_t td = T_ * d, tq = T_ * qkvd, ta = T_ * (size_t)Hq * dh;
    const size_t tu = T_ * (size_t)(gpt2 ? F : 2 * F), tz = T_ * F;
    W.fused = bf16 && !force_unfused && flash_supported(dh, S);
    const bool fused = W.fused;
    const size_t pp = fused ? 0 : (size_t)B * Hq * S * S;   // score-shaped matrices (unfused path only)
    const size_t rows = (size_t)B * Hq * S;
    W.ls.assign(L, LayerSpans{});
    W.rc = recompute;
    // the activations a layer's backward reads (everything but its input pair)
    auto take_acts = [&](LayerSpans& s) {
      take(s.a_m, td * ob); take(s.a_d, td * ob);
      take(s.qkv_m, tq * ob); take(s.qkv_d, tq * ob);
      take(s.P_m, pp * ob); take(s.P_d, pp * ob);
      take(s.st, fused ? rows * 16 : 0);
      take(s.o_m, ta * ob); take(s.o_d, ta * ob);
      take(s.xmid_m, td * 4); take(s.xmid_d, td * 4);
      take(s.b_m, td * ob); take(s.b_d, td * ob);
      take(s.u_m, tu * ob); take(s.u_d, tu * ob);
      take(s.z_m, tz * ob); take(s.z_d, tz * ob);
    };
    for (int l = 0; l < L; ++l) {
      LayerSpans& s = W.ls[l];
      take(s.x_in_m, td * 4); take(s.x_in_d, td * 4);
      if (!W.rc) take_acts(s);
    }
    if (W.rc && L > 0) {
      LayerSpans shared;
      take_acts(shared);
      for (LayerSpans& s : W.ls) {
        const Span xm = s.x_in_m, xd = s.x_in_d;
        s = shared;
        s.x_in_m = xm; s.x_in_d = xd;
      }
    }
    take(W.xL_m, td * 4); take(W.xL_d, td * 4);
    take(W.f_m, td * ob); take(W.f_d, td * ob);
    take(W.lo, (size_t)P * ob);
    take(W.sc_m, pp * 4); take(W.sc_d, pp * 4);
    take(W.log_m, T_ * V * 4); take(W.log_d, T_ * V * 4);
    take(W.dlog_m, T_ * V * ob); take(W.dlog_d, T_ * V * ob);
    take(W.rowloss, 2 * T_ * 8);
    take(W.losses, 2 * 8);
    take(W.tcount, 3 * 8);
    take(W.dx0_m, td * 4); take(W.dx0_d, td * 4);
    take(W.dx1_m, td * 4); take(W.dx1_d, td * 4);
    take(W.dxo_m, td * ob); take(W.dxo_d, td * ob);
    take(W.dz_m, tz * 4); take(W.dz_d, tz * 4);
    take(W.dgu_m, tu * ob); take(W.dgu_d, tu * ob);
    take(W.dudf, gpt2 ? tz * 4 : 0);
    take(W.db_m, td * 4); take(W.db_d, td * 4);
    take(W.gpart, std::max(td * 4, (size_t)2 * norm_bwd_groups((int)T_) * d * 8));
    take(W.do_m, ta * ob); take(W.do_d, ta * ob);
    take(W.dS_m, pp * ob); take(W.dS_d, pp * ob);
    take(W.dqkv_m, tq * 4); take(W.dqkv_d, tq * 4);
    take(W.dqkvo_m, tq * ob); take(W.dqkvo_d, tq * ob);
    take(W.gqa_m, Hq != Hk && !fused ? ta * 4 : 0); take(W.gqa_d, Hq != Hk && !fused ? ta * 4 : 0);
    take(W.dl, fused ? rows * 8 : 0);
    take(W.da_m, td * 4); take(W.da_d, td * 4);
    {
      const int nu = gpt2 ? F : 2 * F;
      size_t mx = 0;
      const int shapes[5][2] = {{qkvd, d}, {d, Hq * dh}, {nu, d}, {d, F}, {V, d}};
      for (const auto& sh : shapes) {
        const int ns = wgrad_splits(sh[0], sh[1], (int)T_);
        if (ns > 1) mx = std::max(mx, (size_t)ns * sh[0] * sh[1] * 4);
      }
      // the down projection's slices when the MLP weight gradients share a launch
      const int nm = bf16 && !gpt2 ? mlp_wgrad_split(nu, d, d, F, (int)T_) : 0;
      if (nm > 1) mx = std::max(mx, (size_t)nm * d * F * 4);
      take(W.wsplit, mx);
    }
    const size_t maxc = std::max<size_t>({(size_t)qkvd, (size_t)F, (size_t)d, (size_t)1});
    take(W.colpart, 64 * maxc * 8);
    take(W.keys, T_ * 4);
    take(W.rope, (size_t)Smax * dh * 8);
    take(W.cdf, (size_t)V * 8);
  }
  take(W.gpartial, 1024 * 8);
  take(W.nfflag, 4 * 4);
  take(W.bpart, 256 * 4 * 8);
  take(W.bout, (size_t)std::max(L, 1) * 4 * 8);
  // Lanczos
  if (m > 0) {
    const int reorth = o ? o->reorth : FDH_REORTH_NONE;
    const int bdt = o ? o->basis_dtype : FDH_F32;
    int cap = 0;
    if (reorth == FDH_REORTH_FULL) cap = m;
    else if (reorth == FDH_REORTH_WINDOW) cap = std::min(m, o->window);
    take(W.lz_w, (size_t)P * 4);
    take(W.lz_q, (size_t)P * 4);
    take(W.lz_qp, (size_t)P * 4);
    const int64_t ldq = (P + 7) / 8 * 8;
    W.lz_ldq = ldq;
    // with the basis offload only the first off_rows rows live in the workspace
    const int ndev = off_rows >= 0 ? std::min(cap, off_rows) : cap;
    W.lz_dev_rows = ndev;
    take(W.lz_basis, (size_t)ndev * ldq * (bdt == FDH_BF16 ? 2 : 4));
    take(W.lz_alpha, (size_t)m * 8);
    take(W.lz_beta, (size_t)m * 8);
    take(W.lz_coef, 128 * 8);
    take(W.lz_gram, 128 * 128 * 8);
    take(W.lz_partial, (size_t)RED_BLOCKS * (2 * cap + 1) * 8);
    take(W.lz_flag, 2 * 4);
    take(W.lz_maxabs, 8);
  }
  W.planB = B;
  W.planS = S;
  W.planM = m;
  if (o) W.planO = *o;
  W.total = cur;
  if (out) *out = std::move(W);
  return cur;
}

int Engine::set_workspace(void* dev, size_t bytes, int B, int S, int m, const fdh_lanczos_opts* o) {
  if (!dev && bytes == 0) {  // detach: the context holds no workspace any more
    static_cast<WsLayout&>(*this) = WsLayout{};
    ws = nullptr;
    ws_bytes = 0;
    lo_for_v = nullptr;
    return FDH_OK;
  }
  if (!dev || B < 0 || S < 0 || m < 0 || (m > 0 && !o)) { err = "bad workspace arguments"; return FDH_ERR_INVALID_ARG; }
  if ((reinterpret_cast<uintptr_t>(dev) & (ALIGN - 1)) != 0) { err = "workspace must be 256-byte aligned"; return FDH_ERR_WORKSPACE; }
  WsLayout W;
  const size_t need = plan(B, S, m, o, &W);
  if (bytes < need) { err = "workspace smaller than fdh_workspace_bytes"; return FDH_ERR_WORKSPACE; }
  static_cast<WsLayout&>(*this) = std::move(W);
  ws = (char*)dev;
  ws_bytes = bytes;
  // a perturbation operand written into the previous carve is not in this one
  lo_for_v = nullptr;
  return FDH_OK;
}

// FNV-1a over every span, the basis geometry, the attention path and the plan
uint64_t Engine::layout_digest() const {
  uint64_t h = 1469598103934665603ull;
  auto mix = [&](uint64_t x) {
    for (int i = 0; i < 8; ++i) {
      h ^= (x >> (8 * i)) & 0xff;
      h *= 1099511628211ull;
    }
  };
  auto sp = [&](const Span& x) { mix(x.off); mix(x.bytes); };
  for (const LayerSpans& s : ls)
    for (const Span* x : {&s.x_in_m, &s.x_in_d, &s.a_m, &s.a_d, &s.qkv_m, &s.qkv_d, &s.P_m, &s.P_d, &s.st, &s.o_m,
                          &s.o_d, &s.xmid_m, &s.xmid_d, &s.b_m, &s.b_d, &s.u_m, &s.u_d, &s.z_m, &s.z_d})
      sp(*x);
  for (const Span* x : {&xL_m, &xL_d, &f_m, &f_d, &lo, &sc_m, &sc_d, &log_m, &log_d, &dlog_m, &dlog_d, &rowloss,
                        &losses, &dx0_m, &dx0_d, &dx1_m, &dx1_d, &dxo_m, &dxo_d, &dz_m, &dz_d, &dgu_m, &dgu_d, &dudf,
                        &db_m, &db_d, &gpart, &do_m, &do_d, &dS_m, &dS_d, &dqkv_m, &dqkv_d, &dqkvo_m, &dqkvo_d, &gqa_m,
                        &gqa_d, &dl, &da_m, &da_d, &colpart, &keys, &rope, &cdf, &gpartial, &bpart, &bout, &tcount,
                        &nfflag, &wsplit, &lz_w, &lz_q, &lz_qp, &lz_basis, &lz_alpha, &lz_beta, &lz_coef, &lz_gram,
                        &lz_partial, &lz_flag, &lz_maxabs})
    sp(*x);
  mix((uint64_t)lz_ldq);
  mix((uint64_t)lz_dev_rows);
  mix(fused ? 1 : 0);
  mix(rc ? 1 : 0);
  mix((uint64_t)planB);
  mix((uint64_t)planS);
  mix((uint64_t)planM);
  mix((uint64_t)planO.reorth);
  mix((uint64_t)planO.window);
  mix((uint64_t)planO.basis_dtype);
  mix(total);
  mix((uint64_t)(uintptr_t)ws);
  mix(ws_bytes);
  return h;
}

// ---------------------------------------------------------------------------
// launch timing (testing hook)
// ---------------------------------------------------------------------------
hipError_t Timing::begin(hipStream_t s, int* e0) {
  if (ev.empty()) {
    ev.resize(POOL);
    for (auto& x : ev) {
      hipError_t r = hipEventCreate(&x);
      if (r != hipSuccess) return r;
    }
  }
  if (used + 2 > ev.size()) {
    hipError_t r = harvest(s);
    if (r != hipSuccess) return r;
  }
  *e0 = (int)used;
  used += 2;
  return hipEventRecord(ev[*e0], s);
}

hipError_t Timing::end(hipStream_t s, int cat, int e0, double fl, double by) {
  recs.push_back({cat, e0, fl, by});
  return hipEventRecord(ev[e0 + 1], s);
}

hipError_t Timing::harvest(hipStream_t s) {
  hipError_t r = hipStreamSynchronize(s);
  if (r != hipSuccess) return r;
  for (const Rec& x : recs) {
    float t = 0.f;
    r = hipEventElapsedTime(&t, ev[x.e0], ev[x.e0 + 1]);
    if (r != hipSuccess) return r;
    ms[x.cat] += t;
    flops[x.cat] += x.flops;
    bytes[x.cat] += x.bytes;
    count[x.cat] += 1.0;
  }
  recs.clear();
  used = 0;
  return hipSuccess;
}

Timing::~Timing() {
  for (auto& x : ev) (void)hipEventDestroy(x);
}

// executed (tile-exact, tails clipped) FLOPs of one GEMM call
static double gemm_flops(const GemmArgs& g) {
  const int BMt = 128;
  double f = 0.0;
  for (int m0 = 0; m0 < g.M; m0 += BMt) {
    const double rows = std::min(BMt, g.M - m0);
    double cols = g.N, kk = g.K;
    if (g.causal == CAUSAL_SKIP_UPPER) cols = std::min<double>(g.N, m0 + BMt);
    if (g.causal == CAUSAL_K_LE_M) kk = std::min<double>(g.K, m0 + BMt);
    if (g.causal == CAUSAL_K_GE_M) kk = g.K - std::min(m0, g.K);
    f += 2.0 * rows * cols * kk;
  }
  return f * g.npairs * g.nbatch;
}

// ---------------------------------------------------------------------------
// GEMM plumbing
// ---------------------------------------------------------------------------
template <typename T>
static int run_gemm(Engine& e, GemmArgs& g) {
  const char* msg = gemm_check<T>(g);
  if (msg) {
    e.err = msg;
    return FDH_ERR_UNSUPPORTED;
  }
  int e0 = 0;
  if (e.timing.on) {
    hipError_t r = e.timing.begin(e.stream, &e0);
    if (r != hipSuccess) { e.err = "timing event"; return FDH_ERR_HIP; }
  }
  hipError_t r = gemm<T>(g, e.stream);
  if (r != hipSuccess) {
    e.err = std::string("gemm launch: ") + hipGetErrorString(r);
    return FDH_ERR_HIP;
  }
  if (e.timing.on) {
    r = e.timing.end(e.stream, 0, e0, gemm_flops(g), 0.0);
    if (r != hipSuccess) { e.err = "timing event"; return FDH_ERR_HIP; }
  }
  return FDH_OK;
}

template <typename T>
static int run_gemm_pair(Engine& e, GemmArgs& g0, GemmArgs& g1) {
  for (const GemmArgs* g : {&g0, &g1}) {
    const char* msg = gemm_check<T>(*g);
    if (msg) {
      e.err = msg;
      return FDH_ERR_UNSUPPORTED;
    }
  }
  int e0 = 0;
  if (e.timing.on) {
    hipError_t r = e.timing.begin(e.stream, &e0);
    if (r != hipSuccess) { e.err = "timing event"; return FDH_ERR_HIP; }
  }
  hipError_t r = gemm_pair<T>(g0, g1, e.stream);
  if (r != hipSuccess) {
    e.err = std::string("gemm launch: ") + hipGetErrorString(r);
    return FDH_ERR_HIP;
  }
  if (e.timing.on) {
    r = e.timing.end(e.stream, 0, e0, gemm_flops(g0) + gemm_flops(g1), 0.0);
    if (r != hipSuccess) { e.err = "timing event"; return FDH_ERR_HIP; }
  }
  return FDH_OK;
}

#define RG(T, g)                       \
  do {                                 \
    int rc_ = run_gemm<T>(*this, g);   \
    if (rc_ != FDH_OK) return rc_;     \
  } while (0)

// ---------------------------------------------------------------------------
// lockstep FD-HVP
// ---------------------------------------------------------------------------
// One batch of the FD-HVP.  The cross-entropy rows are scaled by inv_n; with
// acc the batch's Hv is added to hv (and its losses to the loss pair), which
// is how several batches form the token-weighted dataset average (Algorithm 1).
template <typename T>
int Engine::hvp_t(const T* th, const float* v, double eps, const int32_t* tok, const int32_t* lab, int B, int S,
                  double inv_n, bool acc, float* hv) {
  hipStream_t st = stream;
  const int T_ = B * S;
  const float feps = (float)eps;
  const float inv_eps = (float)(1.0 / eps);
  const bool ln = gpt2;
  const float neps = cfg.norm_eps;
  const int G = Hq / Hk;
  const float att_scale = (float)(1.0 / std::sqrt((double)dh));
  // fused attention arguments shared by the forward and backward launches
  auto flash_args = [&](const T* qm_, const T* qd_, float scale) {
    FlashArgs fa{};
    fa.qkv_m = (const bf16_t*)qm_; fa.qkv_d = (const bf16_t*)qd_; fa.ld = qkvd;
    fa.S = S; fa.Hq = Hq; fa.Hk = Hk; fa.G = G; fa.D = dh;
    fa.koff = Hq * dh; fa.voff = (Hq + Hk) * dh;
    fa.scale = scale;
    fa.ldo = (int64_t)Hq * dh;
    return fa;
  };
  auto F32 = [&](const Span& s) { return (float*)(ws + s.off); };
  auto OP = [&](const Span& s) { return (T*)(ws + s.off); };
  T* lo = OP(this->lo);
  const int64_t pp_stride = (int64_t)S * S;  // per (b,h) matrix

  // perturbation operand: lo = eps * v in the operand type (unless the
  // Lanczos normalisation already wrote it for this v and eps, or an earlier
  // batch of the same product did)
  const bool lo_ready = acc || (lo_for_v == v && lo_for_eps == eps);
  lo_for_v = nullptr;
  int* nf = (int*)(ws + nfflag.off);  // [0] v non-finite, [1] Hv non-finite, [2] token out of range
  if (!lo_ready) CK(launch_scale_cast<T>(lo, v, eps, P, st, nf));
  if (llama) CK(launch_rope_table((double*)(ws + rope.off), S, dh, (double)cfg.rope_base, st));

  // ---- linear helpers ----
  // Y = X W^T (+ bias) (+ residual R, fp32 output only) at both points; out:
  // fp32 (residual stream, logits) or the operand type (q/k/v and the MLP
  // input product, which only feed operand-type consumers)
  auto lin_fwd = [&](const T* Xm, const T* Xd, int K, const ParamRef& W, const ParamRef& bias, void* Ym, void* Yd,
                     const float* Rm, const float* Rd, int N, int out) -> int {
    GemmArgs g;
    g.M = T_; g.N = N; g.K = K;
    g.A[0] = kmaj(Xm, K);
    g.B[0] = kmaj(th + W.off, K);
    g.C = Ym; g.ldc = N; g.out_type = out;
    g.resid = Rm;
    if (bias.valid()) g.bias_theta = th + bias.off;
    RG(T, g);
    GemmArgs h;
    h.M = T_; h.N = N; h.K = K; h.npairs = 2;
    h.A[0] = kmaj(Xd, K); h.B[0] = kmaj(th + W.off, K);
    h.A[1] = kmaj(Xm, K); h.B[1] = kmaj(lo + W.off, K);
    h.C = Yd; h.ldc = N; h.out_type = out;
    h.resid = Rd;
    if (bias.valid()) { h.bias_v = v + bias.off; h.bias_v_scale = feps; }
    RG(T, h);
    return FDH_OK;
  };
  // dX = dY W ; W [N, K]
  auto lin_dgrad = [&](const T* dYm, const T* dYd, int N, const ParamRef& W, int K, void* dXm, void* dXd, int out) -> int {
    GemmArgs g;
    g.M = T_; g.N = K; g.K = N;
    g.A[0] = kmaj(dYm, N);
    g.B[0] = mnmaj(th + W.off, K);
    g.C = dXm; g.ldc = K; g.out_type = out;
    RG(T, g);
    GemmArgs h;
    h.M = T_; h.N = K; h.K = N; h.npairs = 2;
    h.A[0] = kmaj(dYd, N); h.B[0] = mnmaj(th + W.off, K);
    h.A[1] = kmaj(dYm, N); h.B[1] = mnmaj(lo + W.off, K);
    h.C = dXd; h.ldc = K; h.out_type = out;
    RG(T, h);
    return FDH_OK;
  };
  // Hv_W = (dY.m^T X.d + dY.d^T X.m) / eps
  // (with ns > 1 the token range is cut into ns slices, one GEMM batch entry
  // each, into fp32 partial products that a second pass adds in slice order)
  auto wgrad_args = [&](const T* dYm, const T* dYd, int N, const T* Xm, const T* Xd, int K, const ParamRef& W) {
    GemmArgs g;
    g.M = N; g.N = K; g.K = T_; g.npairs = 2;
    g.A[0] = mnmaj(dYm, N); g.B[0] = mnmaj(Xd, K);
    g.A[1] = mnmaj(dYd, N); g.B[1] = mnmaj(Xm, K);
    g.C = hv + W.off; g.ldc = K; g.alpha = inv_eps;
    return g;
  };
  // two weight gradients in one launch, the first over the whole token range,
  // the second (parameter block W1) over ns token slices into fp32 partial
  // products that a second pass adds in slice order
  auto lin_wgrad_pair = [&](GemmArgs g0, GemmArgs g1, int ns, const ParamRef& W1) -> int {
    if (acc) g0.beta = 1.f;
    if (ns <= 1) {
      if (acc) g1.beta = 1.f;
      return run_gemm_pair<T>(*this, g0, g1);
    }
    const int kc = T_ / ns;
    g1.K = kc;
    g1.nbatch = ns;
    for (int p = 0; p < 2; ++p) {
      g1.A[p].s_outer = (int64_t)kc * g1.M;
      g1.B[p].s_outer = (int64_t)kc * g1.N;
    }
    g1.C = F32(wsplit); g1.c_outer = (int64_t)g1.M * g1.N;
    const int rc = run_gemm_pair<T>(*this, g0, g1);
    if (rc != FDH_OK) return rc;
    int e0 = 0;
    if (timing.on) CK(timing.begin(st, &e0));
    CK(launch_sum_splits(hv + W1.off, F32(wsplit), ns, (int64_t)g1.M * g1.N, acc, st));
    if (timing.on) CK(timing.end(st, 0, e0, 0.0, 0.0));
    return FDH_OK;
  };
  auto lin_wgrad = [&](const T* dYm, const T* dYd, int N, const T* Xm, const T* Xd, int K, const ParamRef& W) -> int {
    GemmArgs g = wgrad_args(dYm, dYd, N, Xm, Xd, K, W);
    const int ns = wgrad_splits(N, K, T_);
    if (ns == 1 || force_unsplit || wsplit.bytes < (size_t)ns * N * K * 4) {
      if (acc) g.beta = 1.f;
      RG(T, g);
      return FDH_OK;
    }
    const int kc = T_ / ns;
    g.K = kc;
    g.nbatch = ns;
    for (int p = 0; p < 2; ++p) {
      g.A[p].s_outer = (int64_t)kc * N;
      g.B[p].s_outer = (int64_t)kc * K;
    }
    g.C = F32(wsplit); g.c_outer = (int64_t)N * K;
    RG(T, g);
    int e0 = 0;
    if (timing.on) CK(timing.begin(st, &e0));
    CK(launch_sum_splits(hv + W.off, F32(wsplit), ns, (int64_t)N * K, acc, st));
    if (timing.on) CK(timing.end(st, 0, e0, 0.0, 0.0));
    return FDH_OK;
  };
  auto colsum_hv = [&](const float* X, int C, int64_t ld, const ParamRef& R) -> int {
    CK(launch_colsum(hv + R.off, X, T_, C, ld, 1.0 / eps, acc, (double*)(ws + colpart.off), st));
    return FDH_OK;
  };
  bool op_ready = false;  // dxo holds the operand-type copy of the last norm backward's output
  // norm backward at both points into (dym, dyd) with its operand-type copy in
  // dxo (bf16 models), then the gain (and LayerNorm bias) gradients
  auto norm_back = [&](float* ym, float* yd, const float* rm, const float* rd, const float* xm_, const float* xd_,
                       const float* gm_, const float* gd_, const ParamRef& gain, const ParamRef& bias) -> int {
    const int nwg = norm_bwd_groups(T_);
    double* gp = (double*)F32(gpart);
    double* bp = ln ? gp + (int64_t)nwg * d : nullptr;
    const PairT<T> yo = bf16 ? PairT<T>{OP(dxo_m), OP(dxo_d)} : PairT<T>{nullptr, nullptr};
    CK(launch_norm_bwd<T>(PairF{ym, yd}, yo, rm, rd, xm_, xd_, gm_, gd_, T_, d, ln, th + gain.off, v + gain.off, eps, neps,
                          gp, bp, st));
    op_ready = bf16;
    double* cp = (double*)(ws + colpart.off);
    CK(launch_colsum_f64(hv + gain.off, gp, nwg, d, 1.0 / eps, acc, cp, st));
    if (ln) CK(launch_colsum_f64(hv + bias.off, bp, nwg, d, 1.0 / eps, acc, cp, st));
    return FDH_OK;
  };
  // fp32 pair -> operand pair (aliases in fp32 mode; skipped when the norm
  // backward that produced the pair already wrote the copy)
  auto as_op = [&](const float* m, const float* dd, const Span& om, const Span& od, int64_t n, T** rm, T** rd) -> int {
    if (!bf16) {
      *rm = (T*)m;
      *rd = (T*)dd;
      return FDH_OK;
    }
    if (op_ready) {
      op_ready = false;
      *rm = OP(om);
      *rd = OP(od);
      return FDH_OK;
    }
    PairT<T> o{OP(om), OP(od)};
    CK(launch_cast_pair<T>(o, m, dd, n, st));
    *rm = o.m;
    *rd = o.d;
    return FDH_OK;
  };
#define RC(x)                     \
  do {                            \
    int rc_ = (x);                \
    if (rc_ != FDH_OK) return rc_; \
  } while (0)

  // ================= forward =================
  {
    PairF x0{F32(ls.empty() ? xL_m : ls[0].x_in_m), F32(ls.empty() ? xL_d : ls[0].x_in_d)};
    CK(launch_embed_fwd<T>(x0, tok, T_, S, d, V, th + wte.off, v + wte.off, gpt2 ? th + wpe.off : nullptr,
                           gpt2 ? v + wpe.off : nullptr, eps, nf + 2, st));
  }
  // one decoder layer's forward from its stored input pair x_in: norm 1, qkv,
  // attention, output projection + residual, norm 2, MLP and, with
  // write_next, the down projection into the next layer's input
  auto layer_fwd = [&](int l, bool write_next) -> int {
    const LayerRefs& R = layers[l];
    LayerSpans& s = ls[l];
    const float* xm = F32(s.x_in_m);
    const float* xd = F32(s.x_in_d);
    // norm 1
    CK(launch_norm_fwd<T>(PairT<T>{OP(s.a_m), OP(s.a_d)}, xm, xd, T_, d, ln, th + R.n1g.off, v + R.n1g.off,
                          ln ? th + R.n1b.off : nullptr, ln ? v + R.n1b.off : nullptr, eps, neps, st));
    // qkv projection
    RC(lin_fwd(OP(s.a_m), OP(s.a_d), d, R.wqkv, R.bqkv, OP(s.qkv_m), OP(s.qkv_d), nullptr, nullptr, qkvd, OUT_OP));
    if (llama)
      CK(launch_rope_inplace<T>(PairT<T>{OP(s.qkv_m), OP(s.qkv_d)}, T_, S, Hq, Hk, dh, (const double*)(ws + rope.off), st));
    if (fused) {
      if constexpr (std::is_same<T, bf16_t>::value) {
        FlashArgs fa = flash_args(OP(s.qkv_m), OP(s.qkv_d), att_scale);
        fa.o_m = OP(s.o_m); fa.o_d = OP(s.o_d);
        fa.stats = (float4*)(ws + s.st.off);
        int e0 = 0;
        if (timing.on) CK(timing.begin(st, &e0));
        CK(launch_flash_fwd(fa, B, st));
        // algorithmic: causal S = q k^T and P v for both passes
        if (timing.on) CK(timing.end(st, 2, e0, 4.0 * B * Hq * (double)S * S * dh, 0.0));
      }
    } else {
      // scores S = q k^T / sqrt(dh), causal
      {
        const T* qm = OP(s.qkv_m);
        const T* qd = OP(s.qkv_d);
        GemmOperand Aq_m = kmaj(qm, qkvd), Aq_d = kmaj(qd, qkvd);
        GemmOperand Bk_m = kmaj(qm + Hq * dh, qkvd), Bk_d = kmaj(qd + Hq * dh, qkvd);
        for (GemmOperand* o : {&Aq_m, &Aq_d}) { o->s_outer = (int64_t)S * qkvd; o->s_inner = dh; }
        for (GemmOperand* o : {&Bk_m, &Bk_d}) { o->s_outer = (int64_t)S * qkvd; o->s_inner = dh; o->inner_div = G; }
        GemmArgs g;
        g.M = S; g.N = S; g.K = dh; g.nbatch = B * Hq; g.inner_count = Hq;
        g.A[0] = Aq_m; g.B[0] = Bk_m;
        g.C = F32(sc_m); g.ldc = S; g.c_outer = (int64_t)Hq * pp_stride; g.c_inner = pp_stride;
        g.alpha = att_scale; g.causal = CAUSAL_SKIP_UPPER;
        RG(T, g);
        GemmArgs h = g;
        h.npairs = 2;
        h.A[0] = Aq_m; h.B[0] = Bk_d;
        h.A[1] = Aq_d; h.B[1] = Bk_m;
        h.C = F32(sc_d);
        RG(T, h);
      }
      CK(launch_attn_softmax<T>(PairT<T>{OP(s.P_m), OP(s.P_d)}, F32(sc_m), F32(sc_d), B * Hq * S, S, st));
      // o = P v
      {
        const T* vm = OP(s.qkv_m) + (Hq + Hk) * dh;
        const T* vd = OP(s.qkv_d) + (Hq + Hk) * dh;
        GemmOperand Ap_m = kmaj(OP(s.P_m), S), Ap_d = kmaj(OP(s.P_d), S);
        for (GemmOperand* o : {&Ap_m, &Ap_d}) { o->s_outer = (int64_t)Hq * pp_stride; o->s_inner = pp_stride; }
        GemmOperand Bv_m = mnmaj(vm, qkvd), Bv_d = mnmaj(vd, qkvd);
        for (GemmOperand* o : {&Bv_m, &Bv_d}) { o->s_outer = (int64_t)S * qkvd; o->s_inner = dh; o->inner_div = G; }
        GemmArgs g;
        g.M = S; g.N = dh; g.K = S; g.nbatch = B * Hq; g.inner_count = Hq;
        g.A[0] = Ap_m; g.B[0] = Bv_m;
        g.C = OP(s.o_m); g.ldc = (int64_t)Hq * dh; g.c_outer = (int64_t)S * Hq * dh; g.c_inner = dh;
        g.out_type = OUT_OP; g.causal = CAUSAL_K_LE_M;
        RG(T, g);
        GemmArgs h = g;
        h.npairs = 2;
        h.A[0] = Ap_m; h.B[0] = Bv_d;
        h.A[1] = Ap_d; h.B[1] = Bv_m;
        h.C = OP(s.o_d);
        RG(T, h);
      }
    }
    // output projection + residual
    RC(lin_fwd(OP(s.o_m), OP(s.o_d), Hq * dh, R.wo, R.bo, F32(s.xmid_m), F32(s.xmid_d), xm, xd, d, OUT_F32));
    // norm 2
    CK(launch_norm_fwd<T>(PairT<T>{OP(s.b_m), OP(s.b_d)}, F32(s.xmid_m), F32(s.xmid_d), T_, d, ln, th + R.n2g.off,
                          v + R.n2g.off, ln ? th + R.n2b.off : nullptr, ln ? v + R.n2b.off : nullptr, eps, neps, st));
    // MLP
    const int nu = gpt2 ? F : 2 * F;
    RC(lin_fwd(OP(s.b_m), OP(s.b_d), d, R.w1, R.b1, OP(s.u_m), OP(s.u_d), nullptr, nullptr, nu, OUT_OP));
    if (gpt2) CK(launch_gelu_fwd<T>(PairT<T>{OP(s.z_m), OP(s.z_d)}, OP(s.u_m), OP(s.u_d), (int64_t)T_ * F, st));
    else CK(launch_swiglu_fwd<T>(PairT<T>{OP(s.z_m), OP(s.z_d)}, OP(s.u_m), OP(s.u_d), T_, F, st));
    // the down projection (+ residual) writes the next layer's input; a
    // recompute stops before it, the stored input is already there
    if (!write_next) return FDH_OK;
    float* nxm = (l + 1 < L) ? F32(ls[l + 1].x_in_m) : F32(xL_m);
    float* nxd = (l + 1 < L) ? F32(ls[l + 1].x_in_d) : F32(xL_d);
    RC(lin_fwd(OP(s.z_m), OP(s.z_d), F, R.w2, R.b2, nxm, nxd, F32(s.xmid_m), F32(s.xmid_d), d, OUT_F32));
    return FDH_OK;
  };
  for (int l = 0; l < L; ++l) RC(layer_fwd(l, true));
  // final norm + head + cross-entropy
  CK(launch_norm_fwd<T>(PairT<T>{OP(f_m), OP(f_d)}, F32(xL_m), F32(xL_d), T_, d, ln, th + nfg.off, v + nfg.off,
                        ln ? th + nfb.off : nullptr, ln ? v + nfb.off : nullptr, eps, neps, st));
  RC(lin_fwd(OP(f_m), OP(f_d), d, head, ParamRef{}, F32(log_m), F32(log_d), nullptr, nullptr, V, OUT_F32));
  CK(launch_ce<T>(PairT<T>{OP(dlog_m), OP(dlog_d)}, (double*)(ws + rowloss.off), F32(log_m), F32(log_d), tok, lab, T_,
                  S, V, inv_n, st));
  CK(launch_loss_sum((double*)(ws + losses.off), (const double*)(ws + rowloss.off), T_, acc, st));

  // ================= backward =================
  // head
  RC(lin_wgrad(OP(dlog_m), OP(dlog_d), V, OP(f_m), OP(f_d), d, head));
  RC(lin_dgrad(OP(dlog_m), OP(dlog_d), V, head, d, F32(db_m), F32(db_d), OUT_F32));
  float* dxm = F32(dx0_m);
  float* dxd = F32(dx0_d);
  float* dym = F32(dx1_m);
  float* dyd = F32(dx1_d);
  RC(norm_back(dxm, dxd, nullptr, nullptr, F32(xL_m), F32(xL_d), F32(db_m), F32(db_d), nfg, nfb));

  // token slices of the down projection's weight gradient when the MLP's two
  // weight gradients share a launch (0: two launches)
  int mlp_split = 0;
  if (std::is_same<T, bf16_t>::value && !gpt2 && !force_unsplit && !force_unpaired) {
    mlp_split = mlp_wgrad_split(2 * F, d, d, F, T_);
    if (mlp_split > 1 && wsplit.bytes < (size_t)mlp_split * d * F * 4) mlp_split = 0;
  }
  for (int l = L - 1; l >= 0; --l) {
    const LayerRefs& R = layers[l];
    LayerSpans& s = ls[l];
    // with recomputation the shared activation set still holds the last
    // layer's forward; every earlier layer refills it from its stored input
    if (rc && l < L - 1) RC(layer_fwd(l, false));
    // ---- MLP ----  (dx = gradient w.r.t. layer output)
    T *gom, *god;
    RC(as_op(dxm, dxd, dxo_m, dxo_d, (int64_t)T_ * d, &gom, &god));
    if (gpt2) RC(colsum_hv(dxd, d, d, R.b2));
    // (with mlp_split > 0 the down projection's weight gradient shares the
    // gate/up one's launch below: gom, god and z stay intact until then)
    if (!mlp_split) RC(lin_wgrad(gom, god, d, OP(s.z_m), OP(s.z_d), F, R.w2));
    RC(lin_dgrad(gom, god, d, R.w2, F, F32(dz_m), F32(dz_d), OUT_F32));
    const int nu = gpt2 ? F : 2 * F;
    if (gpt2) {
      CK(launch_gelu_bwd<T>(PairT<T>{OP(dgu_m), OP(dgu_d)}, F32(dudf), OP(s.u_m), OP(s.u_d), F32(dz_m), F32(dz_d),
                            (int64_t)T_ * F, st));
      RC(colsum_hv(F32(dudf), F, F, R.b1));
    } else {
      CK(launch_swiglu_bwd<T>(PairT<T>{OP(dgu_m), OP(dgu_d)}, OP(s.u_m), OP(s.u_d), F32(dz_m), F32(dz_d), T_, F, st));
    }
    if (mlp_split) {
      RC(lin_wgrad_pair(wgrad_args(OP(dgu_m), OP(dgu_d), nu, OP(s.b_m), OP(s.b_d), d, R.w1),
                        wgrad_args(gom, god, d, OP(s.z_m), OP(s.z_d), F, R.w2), mlp_split, R.w2));
    } else {
      RC(lin_wgrad(OP(dgu_m), OP(dgu_d), nu, OP(s.b_m), OP(s.b_d), d, R.w1));
    }
    RC(lin_dgrad(OP(dgu_m), OP(dgu_d), nu, R.w1, d, F32(db_m), F32(db_d), OUT_F32));
    // norm 2 backward, residual: dy = dx + norm2'(db)
    RC(norm_back(dym, dyd, dxm, dxd, F32(s.xmid_m), F32(s.xmid_d), F32(db_m), F32(db_d), R.n2g, R.n2b));
    std::swap(dxm, dym);
    std::swap(dxd, dyd);
    // ---- attention ----  (dx = gradient w.r.t. x_mid)
    RC(as_op(dxm, dxd, dxo_m, dxo_d, (int64_t)T_ * d, &gom, &god));
    if (gpt2) RC(colsum_hv(dxd, d, d, R.bo));
    // (paired with the q/k/v weight gradient below: gom, god and o stay intact
    // through the fused attention backward)
    const bool pair_o = std::is_same<T, bf16_t>::value && fused && !force_unsplit && !force_unpaired &&
                        pair_wgrads(qkvd, d, d, Hq * dh, T_);
    if (!pair_o) RC(lin_wgrad(gom, god, d, OP(s.o_m), OP(s.o_d), Hq * dh, R.wo));
    RC(lin_dgrad(gom, god, d, R.wo, Hq * dh, OP(do_m), OP(do_d), OUT_OP));
    const T* qm = OP(s.qkv_m);
    const T* qd = OP(s.qkv_d);
    float* gm = F32(dqkv_m);
    float* gd = F32(dqkv_d);
    if (fused) {
      if constexpr (std::is_same<T, bf16_t>::value) {
        FlashArgs fa = flash_args(OP(s.qkv_m), OP(s.qkv_d), att_scale);
        fa.o_m = OP(s.o_m); fa.o_d = OP(s.o_d);
        fa.stats = (float4*)(ws + s.st.off);
        fa.do_m = OP(do_m); fa.do_d = OP(do_d);
        fa.delta = (float2*)(ws + dl.off);
        fa.g_m = gm; fa.g_d = gd; fa.ldg = qkvd;
        int e0 = 0;
        if (timing.on) CK(timing.begin(st, &e0));
        CK(launch_flash_bwd(fa, B, st));
        // algorithmic: causal dP, dV, dQ, dK for both passes (the score recompute is not counted)
        if (timing.on) CK(timing.end(st, 2, e0, 8.0 * B * Hq * (double)S * S * dh, 0.0));
      }
    } else {
      // dP = do v^T
      {
        GemmOperand Ao_m = kmaj(OP(do_m), (int64_t)Hq * dh), Ao_d = kmaj(OP(do_d), (int64_t)Hq * dh);
        for (GemmOperand* o : {&Ao_m, &Ao_d}) { o->s_outer = (int64_t)S * Hq * dh; o->s_inner = dh; }
        GemmOperand Bv_m = kmaj(qm + (Hq + Hk) * dh, qkvd), Bv_d = kmaj(qd + (Hq + Hk) * dh, qkvd);
        for (GemmOperand* o : {&Bv_m, &Bv_d}) { o->s_outer = (int64_t)S * qkvd; o->s_inner = dh; o->inner_div = G; }
        GemmArgs g;
        g.M = S; g.N = S; g.K = dh; g.nbatch = B * Hq; g.inner_count = Hq;
        g.A[0] = Ao_m; g.B[0] = Bv_m;
        g.C = F32(sc_m); g.ldc = S; g.c_outer = (int64_t)Hq * pp_stride; g.c_inner = pp_stride;
        g.causal = CAUSAL_SKIP_UPPER;
        RG(T, g);
        GemmArgs h = g;
        h.npairs = 2;
        h.A[0] = Ao_m; h.B[0] = Bv_d;
        h.A[1] = Ao_d; h.B[1] = Bv_m;
        h.C = F32(sc_d);
        RG(T, h);
      }
      CK(launch_attn_dsoftmax<T>(PairT<T>{OP(dS_m), OP(dS_d)}, OP(s.P_m), OP(s.P_d), F32(sc_m), F32(sc_d), B * Hq * S, S, st));
      // dv = P^T do ; dq = dS k / sqrt(dh) ; dk = dS^T q / sqrt(dh)
      {
        const bool grp = G > 1;
        // helpers for the per-(b,h) outputs
        auto out_into = [&](GemmArgs& g, bool to_tmp) {
          if (to_tmp) {
            g.ldc = (int64_t)Hq * dh; g.c_outer = (int64_t)S * Hq * dh; g.c_inner = dh;
          } else {
            g.ldc = qkvd; g.c_outer = (int64_t)S * qkvd; g.c_inner = dh;
          }
        };
        // dv
        GemmOperand At_m = mnmaj(OP(s.P_m), S), At_d = mnmaj(OP(s.P_d), S);
        for (GemmOperand* o : {&At_m, &At_d}) { o->s_outer = (int64_t)Hq * pp_stride; o->s_inner = pp_stride; }
        GemmOperand Bo_m = mnmaj(OP(do_m), (int64_t)Hq * dh), Bo_d = mnmaj(OP(do_d), (int64_t)Hq * dh);
        for (GemmOperand* o : {&Bo_m, &Bo_d}) { o->s_outer = (int64_t)S * Hq * dh; o->s_inner = dh; }
        const int voff = (Hq + Hk) * dh, koff = Hq * dh;
        {
          GemmArgs g;
          g.M = S; g.N = dh; g.K = S; g.nbatch = B * Hq; g.inner_count = Hq; g.causal = CAUSAL_K_GE_M;
          g.A[0] = At_m; g.B[0] = Bo_m;
          out_into(g, grp);
          g.C = grp ? F32(gqa_m) : gm + voff;
          RG(T, g);
          GemmArgs h = g;
          h.npairs = 2;
          h.A[0] = At_m; h.B[0] = Bo_d;
          h.A[1] = At_d; h.B[1] = Bo_m;
          h.C = grp ? F32(gqa_d) : gd + voff;
          RG(T, h);
          if (grp) {
            CK(launch_group_sum(gm + voff, qkvd, F32(gqa_m), T_, Hk, G, dh, st));
            CK(launch_group_sum(gd + voff, qkvd, F32(gqa_d), T_, Hk, G, dh, st));
          }
        }
        // dq
        {
          GemmOperand As_m = kmaj(OP(dS_m), S), As_d = kmaj(OP(dS_d), S);
          for (GemmOperand* o : {&As_m, &As_d}) { o->s_outer = (int64_t)Hq * pp_stride; o->s_inner = pp_stride; }
          GemmOperand Bk_m = mnmaj(qm + koff, qkvd), Bk_d = mnmaj(qd + koff, qkvd);
          for (GemmOperand* o : {&Bk_m, &Bk_d}) { o->s_outer = (int64_t)S * qkvd; o->s_inner = dh; o->inner_div = G; }
          GemmArgs g;
          g.M = S; g.N = dh; g.K = S; g.nbatch = B * Hq; g.inner_count = Hq; g.causal = CAUSAL_K_LE_M;
          g.alpha = att_scale;
          g.A[0] = As_m; g.B[0] = Bk_m;
          out_into(g, false);
          g.C = gm;
          RG(T, g);
          GemmArgs h = g;
          h.npairs = 2;
          h.A[0] = As_m; h.B[0] = Bk_d;
          h.A[1] = As_d; h.B[1] = Bk_m;
          h.C = gd;
          RG(T, h);
        }
        // dk
        {
          GemmOperand Ast_m = mnmaj(OP(dS_m), S), Ast_d = mnmaj(OP(dS_d), S);
          for (GemmOperand* o : {&Ast_m, &Ast_d}) { o->s_outer = (int64_t)Hq * pp_stride; o->s_inner = pp_stride; }
          GemmOperand Bq_m = mnmaj(qm, qkvd), Bq_d = mnmaj(qd, qkvd);
          for (GemmOperand* o : {&Bq_m, &Bq_d}) { o->s_outer = (int64_t)S * qkvd; o->s_inner = dh; }
          GemmArgs g;
          g.M = S; g.N = dh; g.K = S; g.nbatch = B * Hq; g.inner_count = Hq; g.causal = CAUSAL_K_GE_M;
          g.alpha = att_scale;
          g.A[0] = Ast_m; g.B[0] = Bq_m;
          out_into(g, grp);
          g.C = grp ? F32(gqa_m) : gm + koff;
          RG(T, g);
          GemmArgs h = g;
          h.npairs = 2;
          h.A[0] = Ast_m; h.B[0] = Bq_d;
          h.A[1] = Ast_d; h.B[1] = Bq_m;
          h.C = grp ? F32(gqa_d) : gd + koff;
          RG(T, h);
          if (grp) {
            CK(launch_group_sum(gm + koff, qkvd, F32(gqa_m), T_, Hk, G, dh, st));
            CK(launch_group_sum(gd + koff, qkvd, F32(gqa_d), T_, Hk, G, dh, st));
          }
        }
      }
    }
    {
      if (gpt2) RC(colsum_hv(gd, qkvd, qkvd, R.bqkv));
      CK(launch_qkv_bwd_post<T>(PairT<T>{OP(dqkvo_m), OP(dqkvo_d)}, gm, gd, T_, S, Hq, Hk, dh,
                                (const double*)(ws + rope.off), llama, st));
    }
    if (pair_o)
      RC(lin_wgrad_pair(wgrad_args(OP(dqkvo_m), OP(dqkvo_d), qkvd, OP(s.a_m), OP(s.a_d), d, R.wqkv),
                        wgrad_args(gom, god, d, OP(s.o_m), OP(s.o_d), Hq * dh, R.wo), 1, R.wo));
    else
      RC(lin_wgrad(OP(dqkvo_m), OP(dqkvo_d), qkvd, OP(s.a_m), OP(s.a_d), d, R.wqkv));
    RC(lin_dgrad(OP(dqkvo_m), OP(dqkvo_d), qkvd, R.wqkv, d, F32(da_m), F32(da_d), OUT_F32));
    RC(norm_back(dym, dyd, dxm, dxd, F32(s.x_in_m), F32(s.x_in_d), F32(da_m), F32(da_d), R.n1g, R.n1b));
    std::swap(dxm, dym);
    std::swap(dxd, dyd);
  }
  // embeddings (difference channel of the gradient w.r.t. the embedding output)
  CK(launch_token_sort((uint32_t*)(ws + keys.off), tok, T_, V, st));
  // (GPT-2 ties the embedding to the head, whose gradient is already in hv)
  if (!gpt2 && !acc) CK(launch_fill_f32(hv + wte.off, (int64_t)V * d, 0.f, st));
  CK(launch_embed_bwd(hv + wte.off, (const uint32_t*)(ws + keys.off), dxd, T_, d, 1.0 / eps, gpt2 || acc, st));
  if (gpt2) {
    CK(launch_pos_bwd(hv + wpe.off, dxd, B, S, d, 1.0 / eps, acc, st));
    if (Smax > S && !acc) CK(launch_fill_f32(hv + wpe.off + (int64_t)S * d, (int64_t)(Smax - S) * d, 0.f, st));
  }
  (void)dxm;
  return FDH_OK;
#undef RC
}

int Engine::check_batch(const int32_t* tok, int B, int S) {
  if (!tok) { err = "null tokens"; return FDH_ERR_INVALID_ARG; }
  if (B < 1 || S < 2) { err = "need B >= 1 and S >= 2"; return FDH_ERR_INVALID_ARG; }
  if (!ws) { err = "no workspace"; return FDH_ERR_WORKSPACE; }
  if (B > planB || S > planS || S > Smax) { err = "batch larger than the workspace plan (or S > max_seq)"; return FDH_ERR_WORKSPACE; }
  if ((int64_t)B * S > 16384) { err = "B*S must be <= 16384"; return FDH_ERR_UNSUPPORTED; }
  if (S > 4096) { err = "S must be <= 4096"; return FDH_ERR_UNSUPPORTED; }
  if (S % 8 || dh % 8) { err = "S and head_dim must be multiples of 8"; return FDH_ERR_UNSUPPORTED; }
  if (fused && S % 128) { err = "this workspace uses fused attention: S must be a multiple of 128"; return FDH_ERR_UNSUPPORTED; }
  return FDH_OK;
}

int Engine::hvp(const void* params, const float* v, double eps, const int32_t* tok, int B, int S, float* hv) {
  if (!params || !v || !hv) { err = "null pointer"; return FDH_ERR_INVALID_ARG; }
  if (!(eps > 0.0) || !std::isfinite(eps)) { err = "eps must be positive and finite"; return FDH_ERR_INVALID_ARG; }
  if ((const void*)hv == params || (const void*)hv == (const void*)v) { err = "hv aliases an input"; return FDH_ERR_INVALID_ARG; }
  if (quad) {
    if (!quad_diag) { err = "QUAD_DIAG: call fdh_set_quad_diag first"; return FDH_ERR_STATE; }
    if (bf16) CK(launch_quad_diag_hvp<bf16_t>((const bf16_t*)params, quad_diag, v, eps, hv, P, stream));
    else CK(launch_quad_diag_hvp<float>((const float*)params, quad_diag, v, eps, hv, P, stream));
    return FDH_OK;
  }
  int rc = check_batch(tok, B, S);
  if (rc != FDH_OK) return rc;
  const double inv_n = 1.0 / ((double)B * (S - 1));
  CK(launch_fill_f32((float*)(ws + nfflag.off), 4, 0.f, stream));
  rc = bf16 ? hvp_t<bf16_t>((const bf16_t*)params, v, eps, tok, nullptr, B, S, inv_n, false, hv)
            : hvp_t<float>((const float*)params, v, eps, tok, nullptr, B, S, inv_n, false, hv);
  if (rc != FDH_OK) return rc;
  return finish_checked(hv);
}

// After a product: scan Hv for NaN/Inf, then wait for the stream and turn the
// flags raised on the way (non-finite direction, token out of range,
// non-finite product) into a status.
int Engine::finish_checked(const float* hv) {
  int* nf = (int*)(ws + nfflag.off);
  CK(launch_nonfinite_scan(hv, P, nf + 1, stream));
  int h[4] = {0, 0, 0, 0};
  CK(hipMemcpyAsync(h, nf, sizeof h, hipMemcpyDeviceToHost, stream));
  CK(hipStreamSynchronize(stream));
  if (h[2]) { err = "a token lies outside [0, vocab)"; return FDH_ERR_INVALID_ARG; }
  if (h[0]) { err = "the direction v holds NaN or Inf"; return FDH_ERR_NONFINITE; }
  if (h[1]) { err = "the product Hv holds NaN or Inf"; return FDH_ERR_NONFINITE; }
  return FDH_OK;
}

int Engine::hvp_batches(const void* params, const float* v, double eps, const BatchRef* bt, int nb, double inv_n,
                        float* hv) {
  if (!params || !v || !hv || !bt) { err = "null pointer"; return FDH_ERR_INVALID_ARG; }
  if (nb < 1) { err = "need at least one batch"; return FDH_ERR_INVALID_ARG; }
  if ((const void*)hv == params || (const void*)hv == (const void*)v) { err = "hv aliases an input"; return FDH_ERR_INVALID_ARG; }
  for (int i = 0; i < nb; ++i) {
    const int rc = check_batch(bt[i].tok, bt[i].B, bt[i].S);
    if (rc != FDH_OK) return rc;
  }
  for (int i = 0; i < nb; ++i) {
    const BatchRef& b = bt[i];
    const int rc = bf16 ? hvp_t<bf16_t>((const bf16_t*)params, v, eps, b.tok, b.lab, b.B, b.S, inv_n, i > 0, hv)
                        : hvp_t<float>((const float*)params, v, eps, b.tok, b.lab, b.B, b.S, inv_n, i > 0, hv);
    if (rc != FDH_OK) return rc;
  }
  return FDH_OK;
}

int Engine::bind_batches(const void* params, const BatchRef* bt, int nb, double eps, int reduction, int64_t* targets) {
  if (!params) { err = "null pointer"; return FDH_ERR_INVALID_ARG; }
  if (!(eps > 0.0) || !std::isfinite(eps)) { err = "eps must be positive and finite"; return FDH_ERR_INVALID_ARG; }
  if (reduction != FDH_REDUCE_MEAN && reduction != FDH_REDUCE_SUM) { err = "unknown reduction"; return FDH_ERR_INVALID_ARG; }
  if (quad) {
    if (nb != 0) { err = "QUAD_DIAG takes no batches"; return FDH_ERR_INVALID_ARG; }
    b_params = params;
    b_data.clear();
    b_eps = eps;
    b_inv_n = 1.0;
    b_targets = 0;
    bound = true;
    return FDH_OK;
  }
  if (nb < 1 || !bt) { err = "need at least one batch"; return FDH_ERR_INVALID_ARG; }
  int64_t cnt[1] = {0};
  for (int i = 0; i < nb; ++i) {
    const int rc = check_batch(bt[i].tok, bt[i].B, bt[i].S);
    if (rc != FDH_OK) return rc;
  }
  {
    // count the kept targets, the invalid labels and the invalid tokens on
    // the device (one small launch per batch), then wait for the three integers
    int64_t* dc = (int64_t*)(ws + tcount.off);
    CK(launch_fill_f64((double*)dc, 3, 0.0, stream));
    for (int i = 0; i < nb; ++i) CK(launch_count_targets(dc, bt[i].tok, bt[i].lab, bt[i].B, bt[i].S, V, stream));
    int64_t h[3];
    CK(hipMemcpyAsync(h, dc, sizeof h, hipMemcpyDeviceToHost, stream));
    CK(hipStreamSynchronize(stream));
    if (h[2] != 0) { err = "tokens must be in [0, vocab)"; return FDH_ERR_INVALID_ARG; }
    if (h[1] != 0) { err = "labels must be in [0, vocab) or -100"; return FDH_ERR_INVALID_ARG; }
    cnt[0] = h[0];
  }
  if (cnt[0] == 0) { err = "the batches hold no targets (every label is -100)"; return FDH_ERR_INVALID_ARG; }
  b_params = params;
  b_data.assign(bt, bt + nb);
  b_eps = eps;
  b_targets = cnt[0];
  b_inv_n = reduction == FDH_REDUCE_MEAN ? 1.0 / (double)cnt[0] : 1.0;
  bound = true;
  if (targets) *targets = cnt[0];
  return FDH_OK;
}

int Engine::hvp_bound_async(const float* v, float* hv) {
  if (!bound) { err = "call fdh_bind first"; return FDH_ERR_STATE; }
  if (quad) return hvp(b_params, v, b_eps, nullptr, 0, 0, hv);
  return hvp_batches(b_params, v, b_eps, b_data.data(), (int)b_data.size(), b_inv_n, hv);
}

int Engine::hvp_bound(const float* v, float* hv) {
  if (!bound) { err = "call fdh_bind first"; return FDH_ERR_STATE; }
  if (quad) return hvp(b_params, v, b_eps, nullptr, 0, 0, hv);
  CK(launch_fill_f32((float*)(ws + nfflag.off), 4, 0.f, stream));
  const int rc = hvp_bound_async(v, hv);
  if (rc != FDH_OK) return rc;
  return finish_checked(hv);
}

int Engine::last_losses(double* lp, double* lm) {
  if (quad || !ws) { err = "no losses for this context"; return FDH_ERR_STATE; }
  double h[2];
  CK(hipMemcpyAsync(h, ws + losses.off, 16, hipMemcpyDeviceToHost, stream));
  CK(hipStreamSynchronize(stream));
  if (lp) *lp = h[0];
  if (lm) *lm = h[1];
  return FDH_OK;
}

// ---------------------------------------------------------------------------
// Lanczos (section 4; Appendix C) with device-resident scalars
// ---------------------------------------------------------------------------
template <typename Bt>
int Engine::lanczos_t(int m, uint64_t seed, const fdh_lanczos_opts& o, double* alpha, double* beta, int* steps) {
  hipStream_t st = stream;
  float* w = (float*)(ws + lz_w.off);
  float* q = (float*)(ws + lz_q.off);
  float* qp = (float*)(ws + lz_qp.off);
  lo_for_v = nullptr;
  LanczosDev D;
  D.alpha = (double*)(ws + lz_alpha.off);
  D.beta = (double*)(ws + lz_beta.off);
  D.coef = (double*)(ws + lz_coef.off);
  D.gram = (double*)(ws + lz_gram.off);
  D.partial = (double*)(ws + lz_partial.off);
  D.flag = (int*)(ws + lz_flag.off);
  D.maxabs = (double*)(ws + lz_maxabs.off);
  const int cap = o.reorth == FDH_REORTH_FULL ? m : (o.reorth == FDH_REORTH_WINDOW ? std::min(m, o.window) : 0);
  const double tol = o.breakdown_tol > 0.f ? (double)o.breakdown_tol : 1e-5;
  // stored rows: the first ones in the workspace, the rest (basis offload) in
  // the caller's pinned host memory
  BasisRows<Bt> R;
  R.dev = (Bt*)(ws + lz_basis.off);
  R.host = (Bt*)host_rows_dev;
  R.ndev = std::min(cap, lz_dev_rows);
  R.ldq = lz_ldq;
  if (cap > R.ndev && (!R.host || host_rows_bytes < (size_t)(cap - R.ndev) * (size_t)lz_ldq * sizeof(Bt))) {
    err = "the basis offload needs a host buffer of (stored rows - device rows) * row bytes";
    return FDH_ERR_WORKSPACE;
  }

  CK(launch_fill_f64(D.alpha, m, 0.0, st));
  CK(launch_fill_f64(D.beta, m, 0.0, st));
  CK(launch_fill_f64(D.maxabs, 1, 0.0, st));
  CK(launch_fill_f32((float*)D.flag, 2, 0.f, st));
  CK(launch_fill_f32(qp, P, 0.f, st));
  CK(launch_rademacher(q, P, seed, st));
  if (cap > 0) CK(launch_scale_cast<Bt>(R.row(0), q, 1.0, P, st));  // slot 0 = q_1

  const double bb = sizeof(Bt), Pd = (double)P;
  // one timed vector launch (algorithmic bytes: each operand touched once)
  auto timed = [&](double bytes, auto&& launch) -> int {
    int e0 = 0;
    if (timing.on) CK(timing.begin(st, &e0));
    CK(launch());
    if (timing.on) CK(timing.end(st, 1, e0, 0.0, bytes));
    return FDH_OK;
  };
#define TV(bytes, ...)                                         \
  do {                                                         \
    int rc_ = timed((bytes), [&]() { return (__VA_ARGS__); }); \
    if (rc_ != FDH_OK) return rc_;                             \
  } while (0)
  for (int k = 0; k < m; ++k) {
    int rc = hvp_bound_async(q, w);
    if (rc != FDH_OK) return rc;
    const int nv = std::min(k + 1, cap);
    if (nv > 0) {
      // step A fused into the projection (reads w, q_prev, q and the rows) and
      // formed again in the update (reads w, q_prev, q, the rows, writes w)
      TV((12.0 + nv * bb) * Pd, launch_lanczos_project<Bt>(w, q, qp, R, nv, k % cap, D, k, P, st));
      TV((16.0 + nv * bb) * Pd, launch_lanczos_update<Bt>(w, q, qp, R, nv, D, k, P, st));
    } else {
      TV(16.0 * Pd, launch_lanczos_alpha(w, q, qp, D, k, P, st));
      TV(12.0 * Pd, launch_lanczos_update<Bt>(w, q, nullptr, R, 0, D, k, P, st));
    }
    Bt* row = nullptr;
    if (cap > 0 && k + 1 < m) row = R.row((k + 1) % cap);
    // the next HVP's perturbation operand is written here too
    const bool next_lo = !quad && k + 1 < m;
    const double ob = bf16 ? 2.0 : 4.0;
    if (next_lo && bf16)
      TV((8.0 + (row ? bb : 0.0) + ob) * Pd,
         launch_lanczos_normalise<Bt, bf16_t>(w, qp, row, (bf16_t*)(ws + this->lo.off), b_eps, D, k, tol, P, st));
    else
      TV((8.0 + (row ? bb : 0.0) + (next_lo ? ob : 0.0)) * Pd,
         launch_lanczos_normalise<Bt, float>(w, qp, row, next_lo ? (float*)(ws + this->lo.off) : nullptr, b_eps, D, k, tol, P, st));
    std::swap(q, qp);
    if (next_lo) {
      lo_for_v = q;
      lo_for_eps = b_eps;
    }
  }
#undef TV
  std::vector<double> a(m), b(m);
  int flag[2];
  CK(hipMemcpyAsync(a.data(), D.alpha, m * 8, hipMemcpyDeviceToHost, st));
  CK(hipMemcpyAsync(b.data(), D.beta, m * 8, hipMemcpyDeviceToHost, st));
  CK(hipMemcpyAsync(flag, D.flag, 8, hipMemcpyDeviceToHost, st));
  CK(hipStreamSynchronize(st));
  const int s = flag[0] ? flag[0] : m;
  for (int k = 0; k < m; ++k) {
    alpha[k] = k < s ? a[k] : 0.0;
    beta[k] = k < s ? b[k] : 0.0;
  }
  *steps = s;
  for (int k = 0; k < s; ++k)
    if (!std::isfinite(a[k]) || !std::isfinite(b[k])) { err = "non-finite Lanczos coefficient"; return FDH_ERR_NONFINITE; }
  return s < m ? FDH_BREAKDOWN : FDH_OK;
}

int Engine::lanczos(int m, uint64_t seed, const fdh_lanczos_opts& o, double* alpha, double* beta, int* steps) {
  if (!bound) { err = "call fdh_bind first"; return FDH_ERR_STATE; }
  if (m < 1 || !alpha || !beta || !steps) { err = "bad lanczos arguments"; return FDH_ERR_INVALID_ARG; }
  if (o.reorth < 0 || o.reorth > 2 || (o.reorth == FDH_REORTH_WINDOW && o.window < 1)) { err = "bad reorth options"; return FDH_ERR_INVALID_ARG; }
  if (!ws || m > planM || o.reorth != planO.reorth || o.basis_dtype != planO.basis_dtype ||
      (o.reorth == FDH_REORTH_WINDOW && std::min(m, o.window) > std::min(planM, planO.window))) {
    err = "Lanczos options or m exceed the workspace plan";
    return FDH_ERR_WORKSPACE;
  }
  if (m > 128) { err = "m must be <= 128"; return FDH_ERR_UNSUPPORTED; }
  if (o.basis_dtype == FDH_BF16) return lanczos_t<bf16_t>(m, seed, o, alpha, beta, steps);
  return lanczos_t<float>(m, seed, o, alpha, beta, steps);
}

// Eigen-decomposition of the symmetric tridiagonal T (order n <= 128) by the
// cyclic Jacobi method (Golub and Van Loan, Matrix Computations, section 8.5):
// plane rotations annihilate each off-diagonal entry in turn until the
// off-diagonal mass vanishes.  On return dd holds the eigenvalues and column i
// of z (row-major n x n) the eigenvector of dd[i].
static void tridiag_eig(int n, std::vector<double>& dd, const std::vector<double>& e, std::vector<double>& z) {
  std::vector<double> A((size_t)n * n, 0.0);
  for (int i = 0; i < n; ++i) A[(size_t)i * n + i] = dd[i];
  for (int i = 0; i + 1 < n; ++i) A[(size_t)i * n + i + 1] = A[(size_t)(i + 1) * n + i] = e[i];
  z.assign((size_t)n * n, 0.0);
  for (int i = 0; i < n; ++i) z[(size_t)i * n + i] = 1.0;
  double fro = 0.0;
  for (double x : A) fro += x * x;
  for (int sweep = 0; sweep < 100; ++sweep) {
    double off = 0.0;
    for (int p = 0; p < n; ++p)
      for (int q = p + 1; q < n; ++q) off += A[(size_t)p * n + q] * A[(size_t)p * n + q];
    if (off <= 1e-32 * fro || off == 0.0) break;
    for (int p = 0; p < n; ++p)
      for (int q = p + 1; q < n; ++q) {
        const double apq = A[(size_t)p * n + q];
        if (apq == 0.0) continue;
        const double tau = (A[(size_t)q * n + q] - A[(size_t)p * n + p]) / (2.0 * apq);
        const double t = (tau >= 0 ? 1.0 : -1.0) / (std::fabs(tau) + std::sqrt(1.0 + tau * tau));
        const double c = 1.0 / std::sqrt(1.0 + t * t), s = t * c;
        for (int k = 0; k < n; ++k) {  // A <- A J  (columns p, q)
          const double akp = A[(size_t)k * n + p], akq = A[(size_t)k * n + q];
          A[(size_t)k * n + p] = c * akp - s * akq;
          A[(size_t)k * n + q] = s * akp + c * akq;
        }
        for (int k = 0; k < n; ++k) {  // A <- J^T A  (rows p, q)
          const double apk = A[(size_t)p * n + k], aqk = A[(size_t)q * n + k];
          A[(size_t)p * n + k] = c * apk - s * aqk;
          A[(size_t)q * n + k] = s * apk + c * aqk;
        }
        for (int k = 0; k < n; ++k) {  // z <- z J
          const double zkp = z[(size_t)k * n + p], zkq = z[(size_t)k * n + q];
          z[(size_t)k * n + p] = c * zkp - s * zkq;
          z[(size_t)k * n + q] = s * zkp + c * zkq;
        }
      }
  }
  for (int i = 0; i < n; ++i) dd[i] = A[(size_t)i * n + i];
}

// Ritz-value diagnostics of T_s (ghost eigenvalues after lost orthogonality,
// Theorem 4.1; the spurious-value test of Cullum and Willoughby, 1985): Ritz
// values ascending with their Gauss weights, residual bounds
// beta_{s+1} |U_si|, cluster sizes (chains of gaps <= tol * max|theta|) and
// the spurious flags (simple values that are also eigenvalues of T without
// its first row and column, within tol * max|theta|).
int ritz_diagnostics(const double* alpha, const double* beta, int s, double tol, double* nodes, double* weights,
                     double* resid, int32_t* copies, int32_t* spurious, int32_t* ghosts) {
  if (!alpha || !beta || s < 1 || s > 128 || !(tol >= 0.0)) return FDH_ERR_INVALID_ARG;
  std::vector<double> dd(alpha, alpha + s), e(beta, beta + (s - 1)), z;
  tridiag_eig(s, dd, e, z);
  std::vector<int> idx(s);
  for (int i = 0; i < s; ++i) idx[i] = i;
  std::sort(idx.begin(), idx.end(), [&](int x, int y) { return dd[x] < dd[y]; });
  std::vector<double> lam(s);
  double norm = 0.0;
  for (int i = 0; i < s; ++i) {
    lam[i] = dd[idx[i]];
    norm = std::max(norm, std::fabs(lam[i]));
  }
  const double thr = tol * norm;
  std::vector<int32_t> cp(s, 1);
  int32_t ng = 0;
  for (int i0 = 0, i = 1; i <= s; ++i) {
    if (i == s || lam[i] - lam[i - 1] > thr) {
      for (int k = i0; k < i; ++k) cp[k] = i - i0;
      ng += i - i0 - 1;
      i0 = i;
    }
  }
  std::vector<double> mu;
  if (s > 1) {
    std::vector<double> e2(beta + 1, beta + (s - 1)), z2;
    mu.assign(alpha + 1, alpha + s);
    tridiag_eig(s - 1, mu, e2, z2);
  }
  for (int i = 0; i < s; ++i) {
    const int c = idx[i];
    if (nodes) nodes[i] = lam[i];
    if (weights) weights[i] = z[c] * z[c];                                   // row 0 of the eigenvectors
    if (resid) resid[i] = std::fabs(beta[s - 1]) * std::fabs(z[(size_t)(s - 1) * s + c]);
    if (copies) copies[i] = cp[i];
    if (spurious) {
      double dmin = INFINITY;
      for (double x : mu) dmin = std::min(dmin, std::fabs(x - lam[i]));
      spurious[i] = (cp[i] == 1 && dmin <= thr) ? 1 : 0;
    }
  }
  if (ghosts) *ghosts = ng;
  return FDH_OK;
}

int Engine::set_basis_offload(int device_rows, void* host, size_t bytes) {
  if (device_rows < 0) {
    off_rows = -1;
    host_rows_dev = nullptr;
    host_rows_bytes = 0;
    return FDH_OK;
  }
  if (device_rows > 128) { err = "device_rows must be <= 128"; return FDH_ERR_INVALID_ARG; }
  void* dptr = nullptr;
  if (host) {
    // the kernels take the device-side address of the pinned host memory
    const hipError_t e = hipHostGetDevicePointer(&dptr, host, 0);
    if (e != hipSuccess || !dptr) {
      (void)hipGetLastError();
      err = "host_rows must be pinned host memory mapped for the device (hipHostMalloc)";
      return FDH_ERR_INVALID_ARG;
    }
  }
  off_rows = device_rows;
  host_rows_dev = dptr;
  host_rows_bytes = host ? bytes : 0;
  return FDH_OK;
}

int Engine::slq(int probes, int m, uint64_t seed, const fdh_lanczos_opts& o, double* nodes, double* weights, int* steps,
                double* trace) {
  if (probes < 1 || !nodes || !weights || !steps) { err = "bad slq arguments"; return FDH_ERR_INVALID_ARG; }
  std::vector<double> a(m), b(m);
  double sum_a1 = 0.0;
  int status = FDH_OK;
  for (int j = 0; j < probes; ++j) {
    int s = 0;
    int rc = lanczos(m, seed + (uint64_t)j, o, a.data(), b.data(), &s);
    if (rc < 0) return rc;
    if (rc == FDH_BREAKDOWN) status = FDH_BREAKDOWN;
    steps[j] = s;
    sum_a1 += a[0];
    std::vector<double> dd(a.begin(), a.begin() + s), e(b.begin(), b.begin() + std::max(0, s - 1)), z;
    tridiag_eig(s, dd, e, z);
    // sort ascending with the first eigenvector components
    std::vector<int> idx(s);
    for (int i = 0; i < s; ++i) idx[i] = i;
    std::sort(idx.begin(), idx.end(), [&](int x, int y) { return dd[x] < dd[y]; });
    for (int i = 0; i < m; ++i) {
      nodes[(size_t)j * m + i] = i < s ? dd[idx[i]] : 0.0;
      weights[(size_t)j * m + i] = i < s ? z[(size_t)0 * s + idx[i]] * z[(size_t)0 * s + idx[i]] : 0.0;
    }
  }
  if (trace) *trace = (double)P * sum_a1 / probes;
  return status;
}

// ---------------------------------------------------------------------------
// synthetic inputs and block statistics
// ---------------------------------------------------------------------------
int Engine::init_params(void* params, uint64_t seed) {
  if (!params) { err = "null params"; return FDH_ERR_INVALID_ARG; }
  for (const Entry& e : entries) {
    const int kind = quad ? FDH_PARAM_MATRIX : e.kind;
    if (bf16) CK(launch_init_range<bf16_t>((bf16_t*)params, e.off, e.numel, kind, seed, 0.02, stream));
    else CK(launch_init_range<float>((float*)params, e.off, e.numel, kind, seed, 0.02, stream));
  }
  return FDH_OK;
}

int Engine::make_tokens(int32_t* tok, int B, int S, uint64_t seed, int dist) {
  if (quad || !tok || B < 1 || S < 1) { err = "bad token arguments"; return FDH_ERR_INVALID_ARG; }
  const int64_t n = (int64_t)B * S;
  if (dist == FDH_TOKENS_UNIFORM) {
    CK(launch_tokens_uniform(tok, n, seed, V, stream));
    return FDH_OK;
  }
  if (dist != FDH_TOKENS_ZIPF) { err = "unknown token distribution"; return FDH_ERR_INVALID_ARG; }
  if (!ws) { err = "Zipf tokens need the workspace"; return FDH_ERR_WORKSPACE; }
  std::vector<double> c(V);
  double acc = 0.0;
  for (int k = 0; k < V; ++k) {
    acc += std::pow((double)(k + 1), -1.1);
    c[k] = acc;
  }
  for (int k = 0; k < V; ++k) c[k] /= acc;
  CK(hipMemcpyAsync(ws + cdf.off, c.data(), (size_t)V * 8, hipMemcpyHostToDevice, stream));
  CK(launch_tokens_zipf(tok, n, seed, (const double*)(ws + cdf.off), V, stream));
  CK(hipStreamSynchronize(stream));  // the host cdf buffer goes out of scope
  return FDH_OK;
}

int Engine::random_vector(float* out, uint64_t seed, int kind) {
  if (!out) { err = "null output"; return FDH_ERR_INVALID_ARG; }
  if (kind == FDH_VEC_RADEMACHER) {
    CK(launch_rademacher(out, P, seed, stream));
    return FDH_OK;
  }
  if (kind != FDH_VEC_GAUSSIAN) { err = "unknown vector kind"; return FDH_ERR_INVALID_ARG; }
  if (!ws) { err = "Gaussian vectors need the workspace"; return FDH_ERR_WORKSPACE; }
  CK(launch_gaussian_unit(out, (double*)(ws + gpartial.off), P, seed, stream));
  return FDH_OK;
}

std::vector<int64_t> Engine::layer_ranges() const {
  std::vector<int64_t> ranges(2 * L);
  for (int l = 0; l < L; ++l) {
    int64_t s0 = -1, s1 = -1;
    for (const Entry& e : entries)
      if (e.layer == l) {
        if (s0 < 0) s0 = e.off;
        s1 = e.off + e.numel;
      }
    ranges[2 * l] = s0;
    ranges[2 * l + 1] = s1;
  }
  return ranges;
}

int Engine::block_stats(const float* a, const float* b, double* out) {
  if (quad || !a || !b || !out) { err = "bad block_stats arguments"; return FDH_ERR_INVALID_ARG; }
  if (!ws) { err = "no workspace"; return FDH_ERR_WORKSPACE; }
  std::vector<int64_t> ranges = layer_ranges();
  std::vector<double> h((size_t)L * 4);
  CK(launch_block_stats(a, b, ranges.data(), L, (double*)(ws + bpart.off), (double*)(ws + bout.off), stream));
  CK(hipMemcpyAsync(h.data(), ws + bout.off, (size_t)L * 4 * 8, hipMemcpyDeviceToHost, stream));
  CK(hipStreamSynchronize(stream));
  for (int l = 0; l < L; ++l)
    for (int c = 0; c < 3; ++c) out[3 * l + c] = h[4 * l + c];
  return FDH_OK;
}

// Exp I (section 6): h = H v, and per layer b, h_b = H v^(b) with v masked to
// layer b (not renormalised); statistics of h^(b) against h_b^(b).
// Conjugate gradient (Hestenes-Stiefel) for (H + lam I) x = b on the bound
// operator, x_0 = 0.  r, p and A p live in the Lanczos vector spans; the
// scalars on the device, (p, A p) and (r, r) read back after each step for the
// breakdown and stopping tests.  The direction update also writes the next
// HVP's perturbation operand.
int Engine::cg_solve(const float* b, double lam, int max_iters, double rel_tol, float* x, double* res, int* steps) {
  if (!b || !x || !res || !steps || max_iters < 0 || !(rel_tol >= 0.0) || !std::isfinite(lam)) {
    err = "bad cg arguments";
    return FDH_ERR_INVALID_ARG;
  }
  if ((const void*)b == (const void*)x) { err = "x aliases b"; return FDH_ERR_INVALID_ARG; }
  if (!bound) { err = "call fdh_bind first"; return FDH_ERR_STATE; }
  if (!ws || planM < 1) { err = "cg needs a workspace planned with m >= 1"; return FDH_ERR_WORKSPACE; }
  hipStream_t st = stream;
  float* r = (float*)(ws + lz_w.off);
  float* p = (float*)(ws + lz_q.off);
  float* ap = (float*)(ws + lz_qp.off);
  double* sc = (double*)(ws + lz_coef.off);
  double* part = (double*)(ws + lz_partial.off);
  const double Pd = (double)P, ob = bf16 ? 2.0 : 4.0;
  for (int k = 0; k <= max_iters; ++k) res[k] = 0.0;
  *steps = 0;
  lo_for_v = nullptr;
  auto timed = [&](double bytes, auto&& launch) -> int {
    int e0 = 0;
    if (timing.on) CK(timing.begin(st, &e0));
    CK(launch());
    if (timing.on) CK(timing.end(st, 1, e0, 0.0, bytes));
    return FDH_OK;
  };
  auto scalar = [&](int i, double* out) -> int {
    CK(hipMemcpyAsync(out, sc + i, 8, hipMemcpyDeviceToHost, st));
    CK(hipStreamSynchronize(st));
    return FDH_OK;
  };
#define TC(bytes, ...)                                         \
  do {                                                         \
    int rc_ = timed((bytes), [&]() { return (__VA_ARGS__); }); \
    if (rc_ != FDH_OK) return rc_;                             \
  } while (0)
  TC(16.0 * Pd, launch_cg_init(x, r, p, b, sc, part, P, st));
  double rr = 0.0;
  int rc = scalar(0, &rr);
  if (rc != FDH_OK) return rc;
  const double bnorm = std::sqrt(rr);
  res[0] = bnorm;
  if (!std::isfinite(bnorm)) { err = "non-finite right-hand side"; return FDH_ERR_NONFINITE; }
  for (int k = 0; k < max_iters; ++k) {
    rc = hvp_bound_async(p, ap);
    if (rc != FDH_OK) return rc;
    TC(12.0 * Pd, launch_cg_ap(ap, p, lam, sc, part, P, st));
    double pap = 0.0;
    rc = scalar(1, &pap);
    if (rc != FDH_OK) return rc;
    if (!std::isfinite(pap)) { err = "non-finite (p, A p)"; return FDH_ERR_NONFINITE; }
    if (!(pap > 0.0)) return FDH_BREAKDOWN;
    TC(24.0 * Pd, launch_cg_step(x, r, p, ap, sc, part, P, st));
    double rn = 0.0;
    rc = scalar(3, &rn);
    if (rc != FDH_OK) return rc;
    res[k + 1] = std::sqrt(rn);
    *steps = k + 1;
    if (!std::isfinite(rn)) { err = "non-finite residual"; return FDH_ERR_NONFINITE; }
    if (res[k + 1] <= rel_tol * bnorm || k + 1 == max_iters) break;
    const bool next_lo = !quad;
    if (next_lo && bf16)
      TC((12.0 + ob) * Pd, launch_cg_dir<bf16_t>(p, r, sc, (bf16_t*)(ws + this->lo.off), b_eps, P, st));
    else
      TC((12.0 + (next_lo ? ob : 0.0)) * Pd,
         launch_cg_dir<float>(p, r, sc, next_lo ? (float*)(ws + this->lo.off) : nullptr, b_eps, P, st));
    if (next_lo) {
      lo_for_v = p;
      lo_for_eps = b_eps;
    }
  }
#undef TC
  return FDH_OK;
}

int Engine::block_diagonal(const float* v, double* out) {
  if (quad || !v || !out) { err = "bad block_diagonal arguments"; return FDH_ERR_INVALID_ARG; }
  if (!bound) { err = "call fdh_bind first"; return FDH_ERR_STATE; }
  if (!ws || planM < 1) { err = "block_diagonal needs a workspace planned with m >= 1"; return FDH_ERR_WORKSPACE; }
  float* h = (float*)(ws + lz_w.off);
  float* vb = (float*)(ws + lz_q.off);
  float* hb = (float*)(ws + lz_qp.off);
  int rc = hvp_bound_async(v, h);
  if (rc != FDH_OK) return rc;
  std::vector<int64_t> ranges = layer_ranges();
  std::vector<double> s4(4);
  for (int l = 0; l < L; ++l) {
    CK(launch_mask_range(vb, v, ranges[2 * l], ranges[2 * l + 1], P, stream));
    rc = hvp_bound_async(vb, hb);
    if (rc != FDH_OK) return rc;
    CK(launch_block_stats(h, hb, &ranges[2 * l], 1, (double*)(ws + bpart.off), (double*)(ws + bout.off), stream));
    CK(hipMemcpyAsync(s4.data(), ws + bout.off, 32, hipMemcpyDeviceToHost, stream));
    CK(hipStreamSynchronize(stream));
    const double na = std::sqrt(s4[0]), nb = std::sqrt(s4[1]), dif = std::sqrt(s4[3]);
    out[4 * l + 0] = dif;
    out[4 * l + 1] = na > 0 ? dif / na : 0.0;
    out[4 * l + 2] = (na > 0 && nb > 0) ? s4[2] / (na * nb) : 0.0;
    out[4 * l + 3] = na;
    for (int c = 0; c < 4; ++c)
      if (!std::isfinite(s4[c])) { err = "non-finite block statistic (NaN or Inf in v or in a product)"; return FDH_ERR_NONFINITE; }
  }
  return FDH_OK;
}

}  // namespace fdh
