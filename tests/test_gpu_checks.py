"""Error paths of the boundary, forced from the host (every kernel still runs
to its end): a NaN or an infinity in the direction v, a non-finite product, a
token outside [0, vocab), and a workspace-size query between two products."""
import numpy as np
import pytest

import synth
from tests.gpu_util import need_gpu, say, upload_params, workload_inputs

pytestmark = pytest.mark.gpu

W = dict(family="llama", n_layers=2, d_model=128, n_heads=8, n_kv_heads=2, d_ff=200, vocab=264, max_seq=128,
         rope_base=10000.0, batch=2, seq=128, token_dist="zipf", dtype="bf16")


def _setup(torch, fd, w=W):
    cfg, theta, tok = workload_inputs(w)
    mod = fd.Model.from_workload(w)
    mod.set_workspace(w["batch"], w["seq"], 2, fd.opts("full", 0, "f32"))
    th = upload_params(torch, theta, w["dtype"])
    dt = torch.from_numpy(tok).cuda()
    v = torch.from_numpy(synth.rademacher_probe(3, theta.size)).cuda()
    return mod, th, dt, v


@pytest.mark.parametrize("bad", [float("nan"), float("inf"), -float("inf")])
def test_nonfinite_direction_is_reported(bad):
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    say(f"non-finite v entry {bad}")
    mod, th, dt, v = _setup(torch, fd)
    good = mod.hvp(th, v, 1e-3, dt).clone()
    vb = v.clone()
    vb[mod.num_params // 3] = bad
    with pytest.raises(fd.FdhError) as e:
        mod.hvp(th, vb, 1e-3, dt)
    assert e.value.status == -4 and "direction" in str(e.value)
    # the flags start from zero at the next call: the same product as before
    again = mod.hvp(th, v, 1e-3, dt)
    assert torch.equal(again, good)
    mod.bind(th, dt, 1e-3)
    with pytest.raises(fd.FdhError) as e:
        mod.hvp_bound(vb)
    assert e.value.status == -4
    assert torch.equal(mod.hvp_bound(v), good)


def test_nonfinite_product_is_reported():
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    say("NaN weight -> non-finite product")
    mod, th, dt, v = _setup(torch, fd)
    lay = {e.name: e for e in mod.layout()}
    bad = th.clone()
    bad[lay["h1.wd"].offset + 5] = float("nan")
    with pytest.raises(fd.FdhError) as e:
        mod.hvp(bad, v, 1e-3, dt)
    assert e.value.status == -4 and "product" in str(e.value)


def test_out_of_range_token_is_rejected():
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    mod, th, dt, v = _setup(torch, fd)
    good = mod.hvp(th, v, 1e-3, dt).clone()
    for t in (W["vocab"], -1, 1 << 20):
        say(f"token {t}")
        bt = dt.clone()
        bt[1, 17] = t
        with pytest.raises(fd.FdhError) as e:
            mod.hvp(th, v, 1e-3, bt)
        assert e.value.status == -1 and "token" in str(e.value)
        with pytest.raises(fd.FdhError) as e:
            mod.bind(th, bt, 1e-3)
        assert e.value.status == -1 and "token" in str(e.value)
        with pytest.raises(fd.FdhError) as e:
            mod.bind_dataset(th, [dt, bt], 1e-3)
        assert e.value.status == -1
    # the last token of a row is only an input; it is checked as well
    bt = dt.clone()
    bt[0, -1] = W["vocab"]
    with pytest.raises(fd.FdhError):
        mod.hvp(th, v, 1e-3, bt)
    assert torch.equal(mod.hvp(th, v, 1e-3, dt), good)


def test_workspace_query_between_products():
    """A size query for another shape (here one that would switch the
    attention path) between two products leaves the second product bit for
    bit the first."""
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    mod, th, dt, v = _setup(torch, fd)
    a = mod.hvp(th, v, 1e-3, dt).clone()
    d0 = mod.layout_digest()
    for B, S, m in [(1, 1000, 0), (8, 64, 40), (2, 136, 1)]:
        mod.workspace_bytes(B, S, m, fd.opts("full", 0, "bf16") if m else None)
    assert mod.layout_digest() == d0
    b = mod.hvp(th, v, 1e-3, dt)
    assert torch.equal(a, b)
