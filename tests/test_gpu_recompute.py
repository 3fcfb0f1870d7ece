"""Activation recomputation (fdh_set_recompute): every layer's forward rerun
from its stored input before its backward gives the same bits as the stored
activations, on the fused (bf16, head dim 128 and 64) and unfused (fp32, and
bf16 forced) attention paths and at the full Llama-3-8B size, where it also
makes room for the window-8 Lanczos run at the workload's full length."""
import numpy as np
import pytest

import synth
from oracle import hvp as OH
from synth.workloads import WORKLOADS
from tests.gpu_util import need_gpu, rel_l2, say, upload_params, workload_inputs

pytestmark = pytest.mark.gpu


def _products(torch, fd, w, B, S, recompute, unfused=False, eps=1e-3):
    cfg, theta, tok = workload_inputs(w, batch=B, seq=S)
    mod = fd.Model.from_workload(w)
    if unfused:
        mod.unfused_attention(True)
    mod.set_recompute(recompute)
    mod.set_workspace(B, S)
    th = upload_params(torch, theta, w["dtype"])
    dt = torch.from_numpy(tok).cuda()
    P = theta.size
    outs = []
    for v in (synth.rademacher_probe(3, P), synth.gaussian_direction(4, P).astype(np.float32)):
        outs.append(mod.hvp(th, torch.from_numpy(v).cuda(), eps, dt).cpu().numpy())
    return outs, mod.last_losses(), (cfg, theta, tok)


@pytest.mark.parametrize("name,layers,B,S,unfused", [
    ("llama-1.3b-bf16", 3, 1, 256, False),      # fused attention, head dim 128
    ("llama3-8b-bf16", 2, 1, 256, False),       # grouped-query heads (32 on 8)
    ("gpt2-medium-bf16", 3, 2, 128, False),     # fused attention, head dim 64
    ("llama-1.3b-bf16", 2, 1, 128, True),       # bf16, unfused attention
    ("tiny-gpt2-fp32", 2, 8, 64, False),        # fp32, score matrices in the workspace
])
def test_recompute_same_bits(name, layers, B, S, unfused):
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    w = dict(WORKLOADS[name], n_layers=layers)
    if name == "llama3-8b-bf16":
        w["vocab"] = 4096
    say(f"recompute: {name}, {layers} layers, {B}x{S} tokens{', unfused attention' if unfused else ''}")
    ref, lref, _ = _products(torch, fd, w, B, S, False, unfused)
    got, lgot, (cfg, theta, tok) = _products(torch, fd, w, B, S, True, unfused)
    for a, b in zip(got, ref):
        assert np.array_equal(a, b), float(np.abs(a - b).max())
    assert lgot == lref
    if w["dtype"] == "f32":
        # and against the oracle directly, at the fp32 bar of the parity tests
        want = OH.lm_hvp(cfg, theta, synth.rademacher_probe(3, theta.size).astype(np.float64), 1e-3, tok)
        err = rel_l2(got[0], want)
        say(f"  rel_l2 against the oracle {err:.3e}")
        assert err <= 5e-3


def _dot(torch, x, y, chunk=1 << 28):
    """fp64 dot product of two float32 device vectors, in chunks (no 64 GB copies)."""
    return sum(float(torch.dot(x[i:i + chunk].double(), y[i:i + chunk].double())) for i in range(0, x.numel(), chunk))


def test_recompute_full_8b_and_window_lanczos():
    """The Llama-3-8B workload at full size (1 x 2048 tokens): Hv with
    recomputation equals Hv without, bit for bit; then the workload's own
    window-8 Lanczos plan (m = 30, 248 GB with recomputation) runs its first
    steps, and alpha_1 = q^T H q, alpha_1^2 + beta_2^2 = ||H q||^2 hold for
    the probe q."""
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    w = WORKLOADS["llama3-8b-bf16"]
    B, S = w["batch"], w["seq"]
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    mod = fd.Model.from_workload(w)
    mod.set_workspace(B, S)
    th = mod.init_params(1)
    tok = mod.make_tokens(B, S, 2, "zipf")
    v = mod.random_vector(3, "rademacher")
    hv0 = mod.hvp(th, v, 1e-3, tok)
    l0 = mod.last_losses()
    mod.set_recompute(True)
    n = mod.set_workspace(B, S)
    hv1 = mod.hvp(th, v, 1e-3, tok)
    l1 = mod.last_losses()
    same = bool(torch.equal(hv0, hv1))
    say(f"8B recompute: workspace {n / 1e9:.1f} GB, Hv identical {same}, losses {l0} / {l1}")
    assert same and l0 == l1
    vhv = _dot(torch, v, hv1)
    nhv2 = _dot(torch, hv1, hv1)
    del hv0, hv1, v
    mod.set_workspace(0, 0)
    torch.cuda.empty_cache()
    m = w["m"]
    o = fd.opts("window", w["window"], w["basis"])
    n = mod.set_workspace(B, S, m, o)
    mod.bind(th, tok, 1e-3)
    steps = 3
    al, be, s, st = mod.lanczos(steps, 3, o)
    say(f"8B window-8 Lanczos with recomputation (workspace {n / 1e9:.1f} GB): steps {s}, alpha {al}, beta {be}")
    assert s == steps and np.all(np.isfinite(al)) and np.all(np.isfinite(be))
    assert abs(al[0] - vhv) <= 1e-4 * abs(vhv) + 1e-12
    assert abs(al[0] ** 2 + be[0] ** 2 - nhv2) <= 1e-4 * nhv2


def test_recompute_dataset_operator_same_bits():
    """The token-weighted dataset operator (three batches of different shapes,
    one with ignored targets) and a short Lanczos run on it: with
    recomputation the products and the Lanczos coefficients are the same bits."""
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    w = dict(WORKLOADS["llama-1.3b-bf16"], n_layers=3)
    cfg, theta, _ = workload_inputs(w, batch=1, seq=128)
    shapes = [(1, 256), (2, 128), (1, 128)]
    toks = [synth.tokens(10 + i, B, S, w["vocab"], "zipf") for i, (B, S) in enumerate(shapes)]
    lab = toks[1].copy()
    lab[:, :40] = -100
    out = {}
    for rc in (False, True):
        mod = fd.Model.from_workload(w)
        mod.set_recompute(rc)
        o = fd.opts("full", 0, "bf16")
        mod.set_workspace(2, 256, 4, o)
        th = upload_params(torch, theta, "bf16")
        db = [torch.from_numpy(toks[0]).cuda(), (torch.from_numpy(toks[1]).cuda(), torch.from_numpy(lab).cuda()),
              torch.from_numpy(toks[2]).cuda()]
        n = mod.bind_dataset(th, db, 1e-3)
        v = torch.from_numpy(synth.rademacher_probe(3, theta.size)).cuda()
        hv = mod.hvp_bound(v).cpu().numpy()
        al, be, s, st = mod.lanczos(4, 5, o)
        out[rc] = (n, hv, al, be)
        say(f"recompute={rc}: {n} targets, alpha {al}")
    assert out[False][0] == out[True][0]
    assert np.array_equal(out[False][1], out[True][1])
    assert np.array_equal(out[False][2], out[True][2]) and np.array_equal(out[False][3], out[True][3])
