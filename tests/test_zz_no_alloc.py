"""fdh_block_stats_noalloc (the allocation-free variant of fdh_block_stats)
against fdh_block_stats, through the C ABI: the same kernels in the same
order, so the statistics must agree bit for bit.  Two calls in a row on the
same GPU share the fixed device scratch; the second uses a smaller model and
vector, so left-over partial sums of the first would show."""
import ctypes as C

import numpy as np
import pytest

from tests.gpu_util import need_gpu, say

pytestmark = pytest.mark.gpu

BIG = dict(family="llama", n_layers=6, d_model=256, n_heads=4, n_kv_heads=2, d_ff=512, vocab=1000, max_seq=64,
           rope_base=10000.0, dtype="bf16")
SMALL = dict(family="gpt2", n_layers=2, d_model=64, n_heads=4, n_kv_heads=4, d_ff=128, vocab=96, max_seq=32,
             rope_base=10000.0, dtype="f32")


def _stats(torch, fd, w, seed):
    mod = fd.Model(w["family"], w["n_layers"], w["d_model"], w["n_heads"], w["n_kv_heads"], w["d_ff"], w["vocab"],
                   w["max_seq"], w["dtype"], rope_base=w["rope_base"])
    P = mod.num_params
    g = torch.Generator(device="cuda").manual_seed(seed)
    a = torch.randn(P, device="cuda", generator=g, dtype=torch.float32)
    b = torch.randn(P, device="cuda", generator=g, dtype=torch.float32)
    torch.cuda.synchronize()
    # the allocation-free call first, on a context that has no workspace at all
    out = np.zeros(3 * mod.num_blocks)
    st = fd.lib().fdh_block_stats_noalloc(mod._h, C.c_void_p(a.data_ptr()), C.c_void_p(b.data_ptr()),
                                          out.ctypes.data_as(C.POINTER(C.c_double)))
    assert st == 0, fd.lib().fdh_last_error(mod._h)
    got = out.reshape(-1, 3)
    mod.set_workspace(1, 8)
    want = mod.block_stats(a, b)
    return got, want, mod, a, b


def test_block_stats_noalloc_matches_workspace_version_twice():
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    got1, want1, m1, a1, b1 = _stats(torch, fd, BIG, 1)
    say(f"noalloc call 1: {got1.shape[0]} blocks, ||a_0||^2 {got1[0, 0]:.9e}")
    assert np.array_equal(got1, want1)
    got2, want2, m2, a2, b2 = _stats(torch, fd, SMALL, 2)
    say(f"noalloc call 2: {got2.shape[0]} blocks, ||a_0||^2 {got2[0, 0]:.9e}")
    assert np.array_equal(got2, want2)
    # independent check of the sums themselves (fp64 on the host)
    lay = [e for e in m2.layout() if e.layer >= 0]
    for l in range(m2.num_blocks):
        es = [e for e in lay if e.layer == l]
        s0, s1 = es[0].offset, es[-1].offset + es[-1].numel
        x = a2[s0:s1].double().cpu().numpy()
        y = b2[s0:s1].double().cpu().numpy()
        ref = np.array([x @ x, y @ y, x @ y])
        assert np.allclose(got2[l], ref, rtol=1e-12, atol=0.0)
    # the binding's wrapper reaches the same entry point
    assert np.array_equal(m1.block_stats_noalloc(a1, b1), want1)
