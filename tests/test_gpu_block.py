"""Exp I (block-diagonal hypothesis) through the C ABI against the oracle."""
import numpy as np
import pytest

import synth
from oracle import block as OB
from oracle import hvp as OH
from oracle import model as M
from tests.gpu_util import need_gpu, say, upload_params, workload_inputs
from tests.test_gpu_parity import SMALL

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,dtype", [("llama-gqa", "f32"), ("gpt2-small", "bf16")])
def test_block_diagonal_matches_oracle(name, dtype):
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    w = dict(SMALL[name], dtype=dtype, n_layers=3)
    say(f"block diagonal {name} {dtype}")
    cfg, theta, tok = workload_inputs(w, std=0.05)
    P = theta.size
    v = synth.gaussian_direction(4, P)
    mod = fd.Model.from_workload(w)
    mod.set_workspace(w["batch"], w["seq"], 1, fd.opts("none"))
    th = upload_params(torch, theta, dtype)
    dt = torch.from_numpy(tok).cuda()
    mod.bind(th, dt, 1e-3)
    got = mod.block_diagonal(torch.from_numpy(v.astype(np.float32)).cuda())
    lay = M.layout(cfg)
    blocks = []
    for l in range(cfg.n_layers):
        ents = [e for e in lay if e.layer == l]
        blocks.append((ents[0].offset, ents[-1].offset + ents[-1].numel))
    st, _, _ = OB.run(lambda x: OH.lm_hvp(cfg, theta, x, 1e-3, tok), v.astype(np.float32).astype(np.float64), blocks)
    tol = 5e-3 if dtype == "f32" else 5e-2
    say(f"  gpu rel {got[:, 1]} oracle rel {st['rel']}")
    assert np.allclose(got[:, 0], st["abs"], rtol=tol, atol=tol * np.abs(st["abs"]).max())
    assert np.allclose(got[:, 1], st["rel"], rtol=tol, atol=tol)
    assert np.allclose(got[:, 2], st["cos"], rtol=tol, atol=tol)


def test_block_diagonal_full_gpt2_medium():
    """Exp I at the GPT-2-medium workload's full size (24 layers, 8 x 1024
    tokens, bf16): the statistics are finite, deterministic and consistent
    with one another (rel = abs / ||h^(b)||, |cos| <= 1, and abs^2 >=
    ||h^(b)||^2 (1 - cos^2), the distance from h^(b) to the line through
    h_b^(b)); the summary is printed as the paper's table reports it."""
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    from synth.workloads import WORKLOADS
    w = WORKLOADS["gpt2-medium-bf16"]
    B, S, L = w["batch"], w["seq"], w["n_layers"]
    mod = fd.Model.from_workload(w)
    mod.set_workspace(B, S, 1, fd.opts("none"))
    th = mod.init_params(1)
    tok = mod.make_tokens(B, S, 2, w["token_dist"])
    mod.bind(th, tok, w["eps"][0])
    v = mod.random_vector(synth.workloads.SEED_GAUSS, "gaussian")
    st = mod.block_diagonal(v)
    assert st.shape == (L, 4) and np.all(np.isfinite(st))
    assert np.array_equal(st, mod.block_diagonal(v))
    ab, rel, cos, nh = st[:, 0], st[:, 1], st[:, 2], st[:, 3]
    assert np.all(nh > 0) and np.allclose(rel, ab / nh, rtol=1e-9)
    assert np.all(np.abs(cos) <= 1.0 + 1e-12)
    assert np.all(ab ** 2 >= nh ** 2 * (1.0 - cos ** 2) * (1.0 - 1e-6))
    say(f"gpt2-medium Exp I over {L} blocks: abs {ab.mean():.4g} +- {ab.std():.3g}, "
        f"rel {rel.mean():.4f} +- {rel.std():.4f}, cos {cos.mean():.4f} +- {cos.std():.4f}")
