"""FD-HVP parity at the bf16 workloads' real token batches (full width and
vocabulary, reduced depth), an error-versus-depth sweep at the 1.3B width, and
the small fp32 workload's Lanczos run at its full configuration.

At these sizes one oracle FD-HVP takes minutes, so the oracle's side was
computed beforehand by ``tests/golden/make_scale_fixtures.py`` (which calls
only ``oracle/`` and ``synth``) and kept as a compact record per product:
exact squared norms of every parameter block, the values at 2048 sampled
indices per block, and the block's inner products with 16 seeded Rademacher
sign vectors.  The GPU side recomputes the same inputs from the same seeds and
is compared element by element on the samples, and on every element through
the sign sketches (for a block of error e, the sketch difference has expected
squared norm 16 ||e||^2).  Bar: relative L2 <= 5e-2 (bf16), per block and over
the whole vector; Ritz extremes within 1e-3 relative (fp32).
"""
import os

import numpy as np
import pytest

import synth
from oracle import lanczos as OL
from synth.workloads import SEED_GAUSS, SEED_PARAMS, SEED_PROBE, SEED_TOKENS, WORKLOADS
from tests import micro
from tests.gpu_util import need_gpu, say, upload_params
from oracle import model as M

pytestmark = pytest.mark.gpu

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "scale")
TOL = 5e-2


def _load(name):
    path = os.path.join(GOLD, name + ".npz")
    if not os.path.exists(path):
        pytest.skip(f"oracle record {name} not generated (tests/golden/make_scale_fixtures.py {name})")
    return np.load(path, allow_pickle=False)


def _inputs(w, B, S):
    cfg = micro.cfg_of(w, bf16=w["dtype"] == "bf16")
    P = M.num_params(cfg)
    theta = synth.init_params(M.init_ranges(cfg), P, SEED_PARAMS, bf16=w["dtype"] == "bf16")
    tok = synth.tokens(SEED_TOKENS, B, S, w["vocab"], w["token_dist"])
    return cfg, theta, tok


def _direction(kind, P):
    if kind == "probe":
        return synth.rademacher_probe(SEED_PROBE, P)
    return synth.gaussian_direction(SEED_GAUSS, P).astype(np.float32)


def _compare(torch, mod, hv, rec, kind):
    """Per-block and whole-vector comparison of the device product hv with the
    oracle record; returns (whole-vector sketch error, worst block sampled
    error, worst block sketch error, norm ratio)."""
    names = [str(x) for x in rec["entry_names"]]
    offs, nums = rec["entry_offsets"], rec["entry_numels"]
    norm2 = rec[f"{kind}_norm2"]
    sk_o = rec[f"{kind}_sketch"]                       # [NSKETCH, blocks]
    nsk = int(rec["nsketch"])
    total = float(np.sqrt(norm2.sum()))
    hv64 = hv.double()
    sk_g = np.zeros_like(sk_o)
    for j in range(nsk):
        z = mod.random_vector(int(rec["sketch_seed0"]) + j, "rademacher")
        zs = torch.sign(z).double()
        for i in range(len(names)):
            o, n = int(offs[i]), int(nums[i])
            sk_g[j, i] = float(torch.dot(hv64[o:o + n], zs[o:o + n]))
        del z, zs
    worst_s, worst_k = 0.0, 0.0
    g_norm2 = np.zeros(len(names))
    for i, name in enumerate(names):
        o, n = int(offs[i]), int(nums[i])
        blk = hv64[o:o + n]
        g_norm2[i] = float(torch.dot(blk, blk))
        if np.sqrt(norm2[i]) <= 1e-3 * total:
            continue
        idx = torch.from_numpy(rec[f"idx{i}"].astype(np.int64)).cuda()
        g = blk[idx].cpu().numpy()
        want = rec[f"{kind}_val{i}"]
        es = float(np.linalg.norm(g - want) / np.linalg.norm(want))
        ek = float(np.linalg.norm(sk_g[:, i] - sk_o[:, i]) / np.linalg.norm(sk_o[:, i]))
        en = abs(np.sqrt(g_norm2[i] / norm2[i]) - 1.0)
        worst_s, worst_k = max(worst_s, es), max(worst_k, ek)
        assert es <= TOL and ek <= TOL and en <= TOL, (name, es, ek, en)
    whole = float(np.linalg.norm(sk_g.sum(1) - sk_o.sum(1)) / np.linalg.norm(sk_o.sum(1)))
    ratio = float(np.sqrt(g_norm2.sum() / norm2.sum()))
    return whole, worst_s, worst_k, ratio


def _run_case(name):
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    rec = _load(name)
    L, B, S = int(rec["n_layers"]), int(rec["batch"]), int(rec["seq"])
    w = dict(WORKLOADS[str(rec["workload"])], n_layers=L)
    say(f"{name}: {w['family']} d={w['d_model']} V={w['vocab']} L={L} tokens {B}x{S}")
    cfg, theta, tok = _inputs(w, B, S)
    P = theta.size
    assert P == int(rec["P"])
    lanczos = "alpha1" in rec.files
    mod = fd.Model.from_workload(w)
    o = fd.opts("full", 0, "bf16" if w["dtype"] == "bf16" else "f32")
    mod.set_workspace(B, S, 2 if lanczos else 0, o if lanczos else None)
    th = upload_params(torch, theta, w["dtype"])
    del theta
    dt = torch.from_numpy(tok).cuda()
    eps = float(rec["eps"])
    out = {}
    for kind in [str(k) for k in rec["dirs"]]:
        v = torch.from_numpy(_direction(kind, P)).cuda()
        hv = mod.hvp(th, v, eps, dt)
        del v
        out[kind] = _compare(torch, mod, hv, rec, kind)
        say(f"  {kind}: whole-vector sketch rel L2 {out[kind][0]:.3e}; worst block sampled {out[kind][1]:.3e}, "
            f"sketch {out[kind][2]:.3e}; ||Hv|| ratio {out[kind][3]:.6f}")
        assert out[kind][0] <= TOL and abs(out[kind][3] - 1.0) <= TOL
        del hv
    if lanczos:
        mod.bind(th, dt, eps)
        a, b, s, _ = mod.lanczos(2, SEED_PROBE, o)
        a1, b2 = float(rec["alpha1"]), float(rec["beta2"])
        nhv = float(np.sqrt(rec["probe_norm2"].sum()))
        say(f"  Lanczos: alpha_1 {a[0]:.6e} vs {a1:.6e}; beta_2 {b[0]:.6e} vs {b2:.6e} (||H q_1|| {nhv:.6e})")
        assert abs(a[0] - a1) <= TOL * nhv
        assert abs(b[0] - b2) <= TOL * b2
    return out


@pytest.mark.parametrize("name", ["llama-1.3b-2l-4x2048", "gpt2-medium-2l-8x1024", "llama3-8b-2l-1x2048"])
def test_hvp_parity_real_token_batch(name):
    _run_case(name)


@pytest.mark.parametrize("depth", [1, 2, 4, 8, 16, 24])
def test_hvp_error_versus_depth_1_3b(depth):
    """The 1.3B width at 1 x 2048 tokens with 1, 2, 4, 8, 16 and 24 layers
    (24: the whole 1.3B model): the bf16 error of the lockstep product,
    recorded against depth."""
    out = _run_case(f"llama-1.3b-depth{depth}-1x2048")
    say(f"  depth {depth}: rel L2 (sketch) {out['probe'][0]:.3e}")


def test_lanczos_small_gpt2_full_config_against_oracle():
    """The small fp32 workload at its full size (16 x 512 tokens, 23.4M
    parameters): one probe, m = 80 steps with full reorthogonalisation and an
    fp32 basis, eps = 1e-3, against the oracle's run of the same 80 steps."""
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    rec = _load("small-gpt2-lanczos-m80")
    w = WORKLOADS["small-gpt2-fp32"]
    m = int(rec["m"])
    cfg, theta, tok = _inputs(w, w["batch"], w["seq"])
    mod = fd.Model.from_workload(w)
    o = fd.opts("full", 0, "f32")
    mod.set_workspace(w["batch"], w["seq"], m, o)
    th = upload_params(torch, theta, "f32")
    dt = torch.from_numpy(tok).cuda()
    mod.bind(th, dt, float(rec["eps"]))
    a, b, s, st = mod.lanczos(m, SEED_PROBE, o)
    ao, bo = rec["alpha"], rec["beta"]
    assert s == m == len(ao)
    lg, wg = OL.ritz(a, b)
    lo, wo = OL.ritz(ao, bo)
    scale = np.abs(lo).max()
    say(f"small-gpt2 m={m}: lambda_max {lg[-1]:.8e} vs {lo[-1]:.8e}; lambda_min {lg[0]:.8e} vs {lo[0]:.8e}; "
        f"alpha_1 {a[0]:.8e} vs {ao[0]:.8e}")
    assert abs(lg[-1] - lo[-1]) <= 1e-3 * scale
    assert abs(lg[0] - lo[0]) <= 1e-3 * scale
    assert abs(a[0] - ao[0]) <= 1e-4 * scale
    say(f"  Gauss weights of the extremes {wg[-1]:.6e} / {wo[-1]:.6e}, {wg[0]:.6e} / {wo[0]:.6e}")
