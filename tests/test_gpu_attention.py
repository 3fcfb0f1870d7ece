"""Fused attention kernels against the unfused attention path on the GPU, and
the token-sliced weight gradients against whole-range ones.

The unfused path (score/probability matrices through the GEMM and row
kernels) is itself pinned to the fp64 oracle by the parity tests; here the
fused kernels (forward, dQ, dK/dV) must reproduce its HVP on the same inputs
to within bf16 rounding, per parameter block, at the workloads' head layouts:
head dimension 128 (Llama 1.3B), 64 (GPT-2 medium) and grouped keys/values
(Llama-3 8B: 32 query heads on 8 key/value heads).  The oracle comparison of
the fused path itself runs in the parity tests, which use it for bf16 models.
"""
import numpy as np
import pytest

from oracle import model as M
from synth.workloads import WORKLOADS
from tests import micro
from tests.gpu_util import need_gpu, rel_l2, say

pytestmark = pytest.mark.gpu


def _both_paths(w, batch, seq, eps=1e-3):
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    out = []
    for unfused in (False, True):
        mod = fd.Model.from_workload(w)
        mod.unfused_attention(unfused)
        mod.set_workspace(batch, seq)
        th = mod.init_params(1)
        tok = mod.make_tokens(batch, seq, 2, "zipf")
        v = mod.random_vector(3, "rademacher")
        out.append(mod.hvp(th, v, eps, tok).double().cpu().numpy())
        del mod
        torch.cuda.synchronize()
    cfg = micro.cfg_of(w, bf16=True)
    return out[0], out[1], M.layout(cfg)


@pytest.mark.parametrize("name,layers,batch,seq", [
    ("llama-1.3b-bf16", 1, 1, 512),
    ("gpt2-medium-bf16", 2, 2, 256),
    ("llama3-8b-bf16", 1, 1, 384),
])
def test_fused_matches_unfused(name, layers, batch, seq):
    w = dict(WORKLOADS[name], n_layers=layers)
    say(f"fused vs unfused attention: {name}, {layers} layer(s), {batch}x{seq}")
    fused, unfused, layout = _both_paths(w, batch, seq)
    assert np.all(np.isfinite(fused))
    err = rel_l2(fused, unfused)
    say(f"  rel_l2 {err:.3e}")
    assert err <= 2e-2
    for e in layout:
        ref = unfused[e.offset:e.offset + e.numel]
        if e.numel >= 4096 and np.linalg.norm(ref) > 1e-3 * np.linalg.norm(unfused):
            be = rel_l2(fused[e.offset:e.offset + e.numel], ref)
            assert be <= 5e-2, (e.name, be)


def test_fused_rejects_unaligned_sequence():
    """A workspace planned for the fused path refuses S that is not a multiple of 128."""
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    w = dict(WORKLOADS["llama-1.3b-bf16"], n_layers=1)
    mod = fd.Model.from_workload(w)
    mod.set_workspace(1, 256)
    th = mod.init_params(1)
    tok = mod.make_tokens(1, 200, 2, "zipf")
    v = mod.random_vector(3, "rademacher")
    with pytest.raises(fd.FdhError):
        mod.hvp(th, v, 1e-3, tok)
    torch.cuda.synchronize()


def test_wgrad_token_slices_match_whole_range():
    """The three launch forms of the weight gradients on the 1.3B layer at
    4096 tokens: by default the 2048 x 2048 output of wo shares one launch with
    the 6144 x 2048 q/k/v one (192 + 64 tiles); without that it is summed over
    four token slices; the reference is one launch per weight over all tokens.
    Only the order of the fp32 partial sums may differ."""
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    w = dict(WORKLOADS["llama-1.3b-bf16"], n_layers=1)
    say("wgrad launch forms (shared launch, token slices, whole range): llama-1.3b, 1 layer, 2x2048")
    out = []
    for mode in (0, 2, 1):
        mod = fd.Model.from_workload(w)
        mod.set_workspace(2, 2048)
        mod.unsplit_wgrad(mode)
        th = mod.init_params(1)
        tok = mod.make_tokens(2, 2048, 2, "zipf")
        v = mod.random_vector(3, "rademacher")
        out.append(mod.hvp(th, v, 1e-3, tok).double().cpu().numpy())
        del mod
        torch.cuda.synchronize()
    layout = M.layout(micro.cfg_of(w, bf16=True))
    ref = out[2]
    for name, got in (("shared launch", out[0]), ("token slices", out[1])):
        err = rel_l2(got, ref)
        say(f"  {name}: rel_l2 {err:.3e}, identical {bool(np.array_equal(got, ref))}")
        assert err <= 1e-4
        for e in layout:
            r = ref[e.offset:e.offset + e.numel]
            if np.linalg.norm(r) > 1e-3 * np.linalg.norm(ref):
                assert rel_l2(got[e.offset:e.offset + e.numel], r) <= 1e-4, (name, e.name)
    # the forms differ only in the wo block (and not at all for q/k/v and the rest)
    wo = [e for e in layout if e.name.endswith("wo")]
    assert wo
    mask = np.ones(ref.size, bool)
    for e in wo:
        mask[e.offset:e.offset + e.numel] = False
    assert np.array_equal(out[1][mask], ref[mask])
    with pytest.raises(fd.FdhError):
        fd.Model.from_workload(w).unsplit_wgrad(3)