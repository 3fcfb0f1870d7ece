"""CG inverse-HVP solver through the C ABI against the fp64 oracle.

* QUAD_DIAG operator (H = diag(d) exactly): the solution of the damped
  system is b / (d + lam) elementwise, and the residual history follows the
  oracle's CG on the same operator; a length that is not a multiple of 8.
* Negative curvature along b stops the solver at once with FDH_BREAKDOWN.
* The tiny GPT-2 language model: up to four steps against the oracle's CG
  driven by the oracle's own FD-HVP (status, step count, residual norms and
  iterate; with lam = 1 both stop at the same negative-curvature breakdown).
* The 1.3B workload at its bench size: a few damped steps run, stay finite and
  reduce the residual.
"""
import numpy as np
import pytest

import synth
from oracle import cg as OC
from oracle import hvp as OH
from synth.workloads import WORKLOADS
from tests.gpu_util import need_gpu, rel_l2, say, workload_inputs, upload_params

pytestmark = pytest.mark.gpu


def _quad(torch, fd, diag):
    P = diag.size
    mod = fd.Model("quad_diag", quad_n=P)
    mod.set_workspace(0, 0, 1, fd.opts("none"))
    d = torch.from_numpy(diag.astype(np.float32)).cuda()
    th = torch.from_numpy(np.linspace(-1, 1, P).astype(np.float32)).cuda()
    mod.set_quad_diag(d)
    mod.bind(th, None, 1e-3)
    mod._keep += [d, th]
    return mod


def test_cg_quad_diag_solution_and_history():
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    P = 100003
    rng = np.random.default_rng(11)
    diag = rng.uniform(0.5, 4.0, P).astype(np.float32)
    lam = 0.25
    b = synth.gaussian_direction(12, P).astype(np.float32)
    mod = _quad(torch, fd, diag)
    x, res, s, st = mod.cg_solve(torch.from_numpy(b).cuda(), lam, 100, 1e-6)
    assert st == fd.OK
    want = b.astype(np.float64) / (diag.astype(np.float64) + lam)
    got = x.double().cpu().numpy()
    say(f"cg quad: {s} steps, rel_l2 {rel_l2(got, want):.2e}")
    assert rel_l2(got, want) <= 1e-5
    xo, so, reso, sto = OC.cg(lambda v: diag.astype(np.float64) * v, b.astype(np.float64), lam, 100, 1e-6)
    assert sto == OC.OK and abs(s - so) <= 1
    k = min(s, so, 12)
    assert np.allclose(res[:k], reso[:k], rtol=1e-4)
    assert res[s] <= 1e-6 * res[0]


def test_cg_breakdown_on_negative_curvature():
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    P = 5000
    diag = np.full(P, -1.0, np.float32)
    diag[:10] = 2.0
    b = synth.rademacher_probe(3, P).astype(np.float32)
    mod = _quad(torch, fd, diag)
    x, res, s, st = mod.cg_solve(torch.from_numpy(b).cuda(), 0.0, 5, 0.0)
    assert st == fd.BREAKDOWN and s == 0
    assert float(x.abs().max()) == 0.0
    assert abs(res[0] - np.linalg.norm(b.astype(np.float64))) <= 1e-6 * res[0]


def test_cg_tiny_gpt2_against_oracle():
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    w = WORKLOADS["tiny-gpt2-fp32"]
    cfg, theta, tok = workload_inputs(w)
    P = theta.size
    eps, lam, steps = 1e-3, 1.0, 4
    b = synth.gaussian_direction(5, P)
    mod = fd.Model.from_workload(w)
    mod.set_workspace(w["batch"], w["seq"], 1, fd.opts("none"))
    th = upload_params(torch, theta, "f32")
    dt = torch.from_numpy(tok).cuda()
    mod.bind(th, dt, eps)
    x, res, s, st = mod.cg_solve(torch.from_numpy(b.astype(np.float32)).cuda(), lam, steps, 0.0)
    xo, so, reso, sto = OC.cg(lambda v: OH.lm_hvp(cfg, theta, v, eps, tok), b.astype(np.float64), lam, steps, 0.0)
    say(f"cg tiny-gpt2: status {st}/{sto}, steps {s}/{so}, res {res} vs {reso}")
    assert st == sto and s == so
    assert np.allclose(res, reso, rtol=1e-4)
    if s > 0:
        assert rel_l2(x.double().cpu().numpy(), xo) <= 1e-4


def test_cg_full_1_3b_runs_and_reduces_residual():
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    w = WORKLOADS["llama-1.3b-bf16"]
    B, S = w["batch"], w["seq"]
    mod = fd.Model.from_workload(w)
    o = fd.opts("full", 0, "bf16")
    mod.set_workspace(B, S, 8, o)
    th = mod.init_params(1)
    tok = mod.make_tokens(B, S, 2, "zipf")
    mod.bind(th, tok, 1e-3)
    al, be, n, _ = mod.lanczos(8, 3, o)
    from oracle import lanczos as OL
    ritz = np.linalg.eigvalsh(OL.tridiag(al[:n], be[:n]))
    lam = 3.0 * float(np.abs(ritz).max())          # H + lam I positive definite with a wide margin
    b = mod.random_vector(4, "gaussian")
    x, res, s, st = mod.cg_solve(b, lam, 3, 0.0)
    say(f"cg 1.3B: lam {lam:.3e}, steps {s}, res {res}")
    assert st == fd.OK and s == 3
    assert np.all(np.isfinite(res)) and bool(torch.isfinite(x).all())
    assert res[-1] < res[0]
