"""HVP parity at the workloads' real layer shapes (full width, vocabulary and
head layout; reduced depth and token count so the fp64 oracle finishes in
seconds; the 8B vocabulary is cut as well), and at the full small fp32
workload.  Also properties that must hold at the full 1.3B and 8B sizes:
symmetry, and agreement of the Lanczos alpha_1 (and beta_2) with the moments
of the probe under separately computed products."""
import numpy as np
import pytest

import synth
from oracle import hvp as OH
from oracle import model as M
from synth.workloads import WORKLOADS
from tests.gpu_util import need_gpu, rel_l2, say, upload_params, workload_inputs

pytestmark = pytest.mark.gpu


def _parity(w, batch, seq, ndirs=1, eps=1e-3):
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    cfg, theta, tok = workload_inputs(w, batch=batch, seq=seq)
    P = theta.size
    mod = fd.Model.from_workload(w)
    mod.set_workspace(batch, seq)
    th = upload_params(torch, theta, w["dtype"])
    dt = torch.from_numpy(tok).cuda()
    vs = [synth.rademacher_probe(3, P), synth.gaussian_direction(4, P)][:ndirs]
    errs = []
    for v in vs:
        got = mod.hvp(th, torch.from_numpy(v).cuda(), eps, dt).cpu().numpy()
        want = OH.lm_hvp(cfg, theta, v.astype(np.float64), eps, tok)
        errs.append(rel_l2(got, want))
        # per-block agreement as well: every layer block within the same bar
        for e in M.layout(cfg):
            if e.numel >= 4096 and np.linalg.norm(want[e.offset:e.offset + e.numel]) > 1e-3 * np.linalg.norm(want):
                be = rel_l2(got[e.offset:e.offset + e.numel], want[e.offset:e.offset + e.numel])
                assert be <= (5e-3 if w["dtype"] == "f32" else 5e-2), (e.name, be)
    return errs


def test_llama_1_3b_layer_shapes_bf16():
    w = dict(WORKLOADS["llama-1.3b-bf16"], n_layers=1)
    say("llama-1.3b shapes, 1 layer, 1x256 tokens")
    errs = _parity(w, 1, 256)
    say(f"  rel_l2 {errs}")
    assert max(errs) <= 5e-2


def test_llama3_8b_layer_shapes_bf16():
    # full width, MLP and grouped-query head layout (32 query heads on 8
    # key/value heads, RoPE base 5e5); the vocabulary is cut to 4096 so that
    # the fp64 oracle's vectors stay at 2 GB (the full vocabulary runs in the
    # fused-attention test and in the full-size test below)
    w = dict(WORKLOADS["llama3-8b-bf16"], n_layers=1, vocab=4096)
    say("llama3-8b shapes, 1 layer, vocab 4096, 1x128 tokens")
    errs = _parity(w, 1, 128)
    say(f"  rel_l2 {errs}")
    assert max(errs) <= 5e-2


def test_gpt2_medium_layer_shapes_bf16():
    w = dict(WORKLOADS["gpt2-medium-bf16"], n_layers=2)
    say("gpt2-medium shapes, 2 layers, 1x256 tokens")
    errs = _parity(w, 1, 256)
    say(f"  rel_l2 {errs}")
    assert max(errs) <= 5e-2


def test_small_gpt2_fp32_full_workload():
    w = WORKLOADS["small-gpt2-fp32"]
    say("small-gpt2 fp32 full workload 16x512")
    errs = _parity(w, w["batch"], w["seq"])
    say(f"  rel_l2 {errs}")
    assert max(errs) <= 5e-3


def test_full_1_3b_properties():
    """At the bench size: (Hv, w) = (v, Hw) and Lanczos alpha_1 = v^T H v."""
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    w = WORKLOADS["llama-1.3b-bf16"]
    B, S = w["batch"], w["seq"]
    mod = fd.Model.from_workload(w)
    o = fd.opts("full", 0, "bf16")
    mod.set_workspace(B, S, 2, o)
    th = mod.init_params(1)
    tok = mod.make_tokens(B, S, 2, "zipf")
    v = mod.random_vector(3, "rademacher")
    u = mod.random_vector(4, "gaussian")
    hv = mod.hvp(th, v, 1e-3, tok)
    hu = mod.hvp(th, u, 1e-3, tok)
    a = float(torch.dot(u.double(), hv.double()))
    b = float(torch.dot(v.double(), hu.double()))
    # for unit u, v the error of u.Hv is ~ ||dHv|| / sqrt(P) with ||dHv|| <~ 5e-2 ||Hv||
    noise = (float(torch.linalg.vector_norm(hv.double())) + float(torch.linalg.vector_norm(hu.double()))) / np.sqrt(mod.num_params)
    say(f"u.Hv = {a:.6e}, v.Hu = {b:.6e}, noise scale {noise:.3e}")
    assert abs(a - b) <= 5e-2 * max(abs(a), abs(b)) + 5e-2 * noise
    vhv = float(torch.dot(v.double(), hv.double()))
    mod.bind(th, tok, 1e-3)
    al, be, s, _ = mod.lanczos(2, 3, o)
    say(f"v.Hv = {vhv:.6e}, alpha_1 = {al[0]:.6e}")
    assert abs(al[0] - vhv) <= 1e-4 * abs(vhv) + 1e-6
    assert np.all(np.isfinite(hv.cpu().numpy()))


def _dot(torch, x, y, chunk=1 << 28):
    """fp64 dot product of two float32 device vectors, in chunks (no 64 GB copies)."""
    return sum(float(torch.dot(x[i:i + chunk].double(), y[i:i + chunk].double())) for i in range(0, x.numel(), chunk))


def test_full_8b_properties_and_window_lanczos():
    """The Llama-3-8B workload at full depth and size (1 x 2048 tokens, P = 8.03e9):
    (u, Hv) = (v, Hu); then its window-8 Lanczos run (10 steps, so the window
    slides) against the moment identities alpha_1 = q^T H q and
    alpha_1^2 + beta_2^2 = ||H q||^2 of the probe q."""
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    w = WORKLOADS["llama3-8b-bf16"]
    B, S = w["batch"], w["seq"]
    # the window-8 workspace (273 GB) and theta (16 GB) leave 20 GB of the
    # 288 GiB: give back what earlier tests left cached first, so that theta is
    # not carved out of one of their segments
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    mod = fd.Model.from_workload(w)
    P = mod.num_params
    mod.set_workspace(B, S)
    th = mod.init_params(1)
    tok = mod.make_tokens(B, S, 2, "zipf")
    v = mod.random_vector(3, "rademacher")
    u = mod.random_vector(4, "gaussian")
    hv = mod.hvp(th, v, 1e-3, tok)
    hu = mod.hvp(th, u, 1e-3, tok)
    assert bool(torch.isfinite(hv).all()) and bool(torch.isfinite(hu).all())
    a, b = _dot(torch, u, hv), _dot(torch, v, hu)
    nhv, nhu = np.sqrt(_dot(torch, hv, hv)), np.sqrt(_dot(torch, hu, hu))
    noise = (nhv + nhu) / np.sqrt(P)
    say(f"8B: u.Hv = {a:.6e}, v.Hu = {b:.6e}, noise scale {noise:.3e}")
    assert abs(a - b) <= 5e-2 * max(abs(a), abs(b)) + 5e-2 * noise
    vhv = _dot(torch, v, hv)
    del hv, hu, u, v
    mod._ws = None
    torch.cuda.empty_cache()
    m = 10
    o = fd.opts("window", w["window"], "bf16")
    mod.set_workspace(B, S, m, o)
    mod.bind(th, tok, 1e-3)
    al, be, s, st = mod.lanczos(m, 3, o)
    say(f"8B window-8 Lanczos: steps {s}, alpha {al}, beta {be}")
    assert s == m and np.all(np.isfinite(al)) and np.all(np.isfinite(be))
    assert abs(al[0] - vhv) <= 1e-4 * abs(vhv) + 1e-12
    assert abs(al[0] ** 2 + be[0] ** 2 - nhv ** 2) <= 1e-4 * nhv ** 2


def test_eps_sweep_small_gpt2_shapes_fp32():
    """The small fp32 workload's step sweep (1e-4, 1e-3, 1e-2) at its layer
    shapes (2 layers, 4 x 128 tokens): at every step the GPU matches the
    oracle's estimator at the same step, and against a near-exact fp64
    reference (the oracle at step 1e-5) the estimator's O(eps^2) truncation
    (Theorem 3.1) grows about 100x from 1e-3 to 1e-2.  Theorem 3.1's rounding
    term, O(u / eps) for a difference of two fp32 gradients, does not appear:
    the lockstep passes carry the difference in a channel of its own, so its
    fp32 rounding is relative to the difference and the GPU's distance to the
    estimator stays flat (about 1e-6) down to the smallest step."""
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    w = dict(WORKLOADS["small-gpt2-fp32"], n_layers=2)
    cfg, theta, tok = workload_inputs(w, batch=4, seq=128)
    P = theta.size
    mod = fd.Model.from_workload(w)
    mod.set_workspace(4, 128)
    th = upload_params(torch, theta, "f32")
    dt = torch.from_numpy(tok).cuda()
    v = synth.rademacher_probe(3, P).astype(np.float64)
    dv = torch.from_numpy(v.astype(np.float32)).cuda()
    exact = OH.lm_hvp(cfg, theta, v, 1e-5, tok)
    rows = {}
    for eps in (1e-4, 1e-3, 1e-2):
        got = mod.hvp(th, dv, eps, dt).double().cpu().numpy()
        est = OH.lm_hvp(cfg, theta, v, eps, tok)
        rows[eps] = (rel_l2(got, est), rel_l2(got, exact), rel_l2(est, exact))
        say(f"eps {eps:.0e}: gpu vs estimator {rows[eps][0]:.3e}, gpu vs exact {rows[eps][1]:.3e}, "
            f"estimator vs exact {rows[eps][2]:.3e}")
    assert rows[1e-3][0] <= 5e-3 and rows[1e-2][0] <= 5e-3
    # truncation: the estimator's own bias scales as eps^2
    assert 30.0 <= rows[1e-2][2] / rows[1e-3][2] <= 300.0
    # no u / eps growth: the GPU's rounding error does not grow as the step shrinks
    assert max(r[0] for r in rows.values()) <= 1e-5
    assert rows[1e-4][0] <= 3.0 * rows[1e-3][0]


def test_slq_small_gpt2_full_config():
    """The small fp32 workload's SLQ configuration at full size (4 Rademacher
    probes, m = 80, full reorthogonalisation with an fp32 basis, eps = 1e-3):
    Gauss weights sum to one per probe, the trace estimate is P times the mean
    alpha_1, and the extreme Ritz value, which converges first, agrees across
    the four independent probes to 1e-3 relative."""
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    w = WORKLOADS["small-gpt2-fp32"]
    B, S, m, probes = w["batch"], w["seq"], w["m"], w["probes"]
    mod = fd.Model.from_workload(w)
    o = fd.opts(w["reorth"], w["window"], w["basis"])
    mod.set_workspace(B, S, m, o)
    th = mod.init_params(1)
    tok = mod.make_tokens(B, S, 2, w["token_dist"])
    mod.bind(th, tok, 1e-3)
    nodes, weights, steps, trace, st = mod.slq_density(probes, m, synth.workloads.SEED_PROBE, o)
    assert np.all(steps == m)
    assert np.allclose(weights.sum(1), 1.0, atol=1e-9)
    lmax = nodes.max(1)
    lmin = nodes.min(1)
    say(f"small-gpt2 SLQ: lambda_max {lmax}, lambda_min {lmin}, trace {trace:.6e}")
    assert np.abs(lmax - lmax.mean()).max() <= 1e-3 * np.abs(lmax).max()
    alpha1 = []
    for j in range(probes):
        a, b, s, _ = mod.lanczos(1, synth.workloads.SEED_PROBE + j, o)
        alpha1.append(a[0])
    assert abs(trace - mod.num_params * np.mean(alpha1)) <= 1e-9 * abs(trace) + 1e-12
