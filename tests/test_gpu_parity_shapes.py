"""HVP parity at the workloads' real layer shapes (full width, vocabulary and
head layout; reduced depth and token count so the fp64 oracle finishes in
seconds), and at the full small fp32 workload.  Also properties that must
hold at the full 1.3B size: symmetry and agreement of the Lanczos alpha_1
with v^T H v."""
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
                assert be <= (5e-3 if w["dtype"] == "f32" else 1e-1), (e.name, be)
    return errs


def test_llama_1_3b_layer_shapes_bf16():
    w = dict(WORKLOADS["llama-1.3b-bf16"], n_layers=1)
    say("llama-1.3b shapes, 1 layer, 1x256 tokens")
    errs = _parity(w, 1, 256)
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
