"""CPU checks of the C ABI: the library loads, exports every declared symbol,
and its host logic (layout, workspace plan, argument validation) is right.
No call here launches GPU work."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from synth.workloads import WORKLOADS
from oracle import model as M
from tests import micro

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
fd = pytest.importorskip("paper_2602_00816_amd.fdhvp")


def _declared(header):
    src = open(os.path.join(ROOT, "include", header)).read()
    return sorted(set(re.findall(r"\b(fdh_\w+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = fd.lib()
    names = _declared("fdhvp.h") + _declared("fdhvp_testing.h")
    assert len(names) >= 19
    for n in names:
        assert hasattr(lib, n), n
    assert lib.fdh_api_version() == 1


def _model(name):
    w = WORKLOADS[name]
    return fd.Model.from_workload(w)


@pytest.mark.parametrize("name", list(WORKLOADS))
def test_layout_matches_oracle(name):
    m = _model(name)
    ora = M.layout(micro.cfg_of(WORKLOADS[name]))
    lay = m.layout()
    assert m.num_params == M.num_params(micro.cfg_of(WORKLOADS[name]))
    assert [e.name for e in lay] == [e.name for e in ora]
    assert [e.offset for e in lay] == [e.offset for e in ora]
    assert [e.numel for e in lay] == [e.numel for e in ora]
    assert [e.layer for e in lay] == [e.layer for e in ora]
    assert [e.kind for e in lay] == [e.kind for e in ora]
    assert m.num_blocks == WORKLOADS[name]["n_layers"]


def test_workspace_plan_grows_with_batch_and_basis():
    m = _model("llama-1.3b-bf16")
    a = m.workspace_bytes(1, 2048)
    b = m.workspace_bytes(4, 2048)
    assert b > a > 0
    o_full = fd.opts("full", 0, "bf16")
    o_f32 = fd.opts("full", 0, "f32")
    P = m.num_params
    c = m.workspace_bytes(4, 2048, 40, o_full)
    d = m.workspace_bytes(4, 2048, 40, o_f32)
    assert c - b >= 40 * P * 2 + 3 * P * 4
    assert d - c >= 40 * P * 2
    # the 1.3B workload with a 40-vector bf16 basis fits in 288 GB of HBM
    assert c < 280e9


def test_argument_validation_without_gpu_work():
    m = _model("tiny-gpt2-fp32")
    lib = fd.lib()
    h = m._h
    # eps <= 0 and null pointers are rejected before anything is launched
    assert lib.fdh_hvp(h, C.c_void_p(16), C.c_void_p(16), 0.0, C.c_void_p(16), 8, 64, C.c_void_p(32)) == -1
    assert lib.fdh_hvp(h, None, C.c_void_p(16), 1e-3, C.c_void_p(16), 8, 64, C.c_void_p(32)) == -1
    assert lib.fdh_hvp(h, C.c_void_p(16), C.c_void_p(16), float("nan"), C.c_void_p(16), 8, 64, C.c_void_p(32)) == -1
    # no workspace yet
    assert lib.fdh_hvp(h, C.c_void_p(16), C.c_void_p(48), 1e-3, C.c_void_p(16), 8, 64, C.c_void_p(32)) == -2
    assert b"workspace" in lib.fdh_last_error(h)
    # Lanczos before bind
    a = np.zeros(4)
    s = C.c_int32()
    o = fd.opts("full")
    assert lib.fdh_lanczos(h, 4, 1, C.byref(o), a.ctypes.data_as(C.POINTER(C.c_double)),
                           a.ctypes.data_as(C.POINTER(C.c_double)), C.byref(s)) == -5
    # dataset binding: reduction, empty list, and a batch beyond the (absent) plan
    one = (fd.Batch * 1)(fd.Batch(16, 0, 8, 64))
    n = C.c_int64()
    assert lib.fdh_bind_dataset(h, C.c_void_p(16), one, 1, 1e-3, 7, C.byref(n)) == -1
    assert lib.fdh_bind_dataset(h, C.c_void_p(16), one, 0, 1e-3, 0, C.byref(n)) == -1
    assert lib.fdh_bind_dataset(h, C.c_void_p(16), one, 1, 1e-3, 0, C.byref(n)) == -2
    assert lib.fdh_hvp_bound(h, C.c_void_p(16), C.c_void_p(32)) == -5
    # Ritz diagnostics: s outside [1, 128], negative tolerance (host code, no GPU)
    z = np.zeros(4)
    pz = z.ctypes.data_as(C.POINTER(C.c_double))
    assert lib.fdh_ritz_diagnostics(pz, pz, 0, 1e-8, None, None, None, None, None, None) == -1
    assert lib.fdh_ritz_diagnostics(pz, pz, 129, 1e-8, None, None, None, None, None, None) == -1
    assert lib.fdh_ritz_diagnostics(pz, pz, 4, -1.0, None, None, None, None, None, None) == -1
    # bad configurations
    bad = fd.ModelConfig(0, 2, 60, 4, 4, 256, 256, 64, 0, 1e-5, 1e4, 0, 0)   # head_dim 15
    out = C.c_void_p()
    assert lib.fdh_create(C.byref(bad), None, C.byref(out)) == -1
    bad = fd.ModelConfig(1, 2, 64, 4, 3, 256, 256, 64, 0, 1e-5, 1e4, 0, 0)   # 3 does not divide 4
    assert lib.fdh_create(C.byref(bad), None, C.byref(out)) == -1
    bad = fd.ModelConfig(1, 2, 64, 4, 4, 256, 256, 64, 7, 1e-5, 1e4, 0, 0)   # dtype
    assert lib.fdh_create(C.byref(bad), None, C.byref(out)) == -1
    # testing GEMM: K not a multiple of the vector width
    assert lib.fdh_testing_gemm(1, 8, 8, 12, 1, 1, 1, C.c_void_p(256), C.c_void_p(256), None, None,
                                C.c_void_p(256), 0, 1.0, 0, None) == -6


def test_quad_diag_context():
    m = fd.Model("quad_diag", quad_n=1000)
    assert m.num_params == 1000
    assert m.num_blocks == 0


def _fake_workspace(lib, h, B, S, m, o, nbytes=None):
    """Hand the context an aligned address that is never dereferenced here (no
    kernel runs in these tests): set_workspace only plans and records it."""
    need = C.c_size_t()
    assert lib.fdh_workspace_bytes(h, B, S, m, C.byref(o) if o else None, C.byref(need)) == 0
    n = need.value if nbytes is None else nbytes
    return lib.fdh_set_workspace(h, C.c_void_p(1 << 40), n, B, S, m, C.byref(o) if o else None), need.value


def _digest(lib, h):
    out = C.c_uint64()
    assert lib.fdh_testing_layout_digest(h, C.byref(out)) == 0
    return out.value


@pytest.mark.parametrize("name", ["llama-1.3b-bf16", "tiny-gpt2-fp32"])
def test_workspace_queries_leave_the_carve_alone(name):
    """fdh_workspace_bytes is a query and a rejected fdh_set_workspace keeps the
    old buffer: neither may move the spans of the workspace in use (a query
    with another S once switched the attention path and shrank the score
    buffers of the live carve)."""
    lib = fd.lib()
    m = _model(name)
    h = m._h
    w = WORKLOADS[name]
    o = fd.opts("full", 0, "bf16" if w["dtype"] == "bf16" else "f32")
    st, need = _fake_workspace(lib, h, w["batch"], w["seq"], 2, o)
    assert st == 0
    d0 = _digest(lib, h)
    for B, S, mm, oo in [(1, 1000, 0, None), (w["batch"], w["seq"] // 2, 40, o), (2 * w["batch"], 8, 1, fd.opts("window", 3))]:
        n = C.c_size_t()
        assert lib.fdh_workspace_bytes(h, B, S, mm, C.byref(oo) if oo else None, C.byref(n)) == 0
        assert _digest(lib, h) == d0
    # too small: rejected, the carve in use stays
    st, _ = _fake_workspace(lib, h, 2 * w["batch"], w["seq"], 3, o, nbytes=need)
    assert st == -2
    assert _digest(lib, h) == d0
    # unaligned: rejected as well
    assert lib.fdh_set_workspace(h, C.c_void_p((1 << 40) + 64), need * 4, 1, 64, 0, None) == -2
    assert _digest(lib, h) == d0
    # an accepted plan for another shape does change it
    st, _ = _fake_workspace(lib, h, 1, 128, 0, None)
    assert st == 0 and _digest(lib, h) != d0


def _activation_set_bytes(w, B, S, fused):
    """Bytes of one layer's activations other than its input pair, written out
    from the model shapes: the pairs (mean, half-difference) of the norm-1
    output, q/k/v, scores (unfused attention only), attention output, fp32
    mid-layer residual, norm-2 output, MLP input product and MLP activation,
    plus the fused attention's per-row statistics."""
    T, d, F = B * S, w["d_model"], w["d_ff"]
    H, Hk = w["n_heads"], w["n_kv_heads"]
    dh = d // H
    ob = 2 if w["dtype"] == "bf16" else 4
    nu = F if w["family"] == "gpt2" else 2 * F
    elems_op = T * d + T * (H + 2 * Hk) * dh + T * H * dh + T * d + T * nu + T * F
    if not fused:
        elems_op += B * H * S * S
    return 2 * elems_op * ob + 2 * T * d * 4 + (B * H * S * 16 if fused else 0)


@pytest.mark.parametrize("name", ["llama3-8b-bf16", "tiny-gpt2-fp32", "gpt2-medium-bf16"])
def test_recompute_plan_keeps_one_activation_set(name):
    """fdh_set_recompute: the plan keeps each layer's input pair and one shared
    activation set, so the workspace shrinks by exactly L - 1 sets; the mode
    is taken at the next fdh_set_workspace, not before."""
    lib = fd.lib()
    w = WORKLOADS[name]
    m = _model(name)
    h = m._h
    B, S = w["batch"], w["seq"]
    fused = w["dtype"] == "bf16" and S % 128 == 0
    n0 = m.workspace_bytes(B, S)
    st, _ = _fake_workspace(lib, h, B, S, 0, None)
    assert st == 0
    d0 = _digest(lib, h)
    m.set_recompute(True)
    n1 = m.workspace_bytes(B, S)
    assert _digest(lib, h) == d0          # the carve in use keeps its mode
    assert n0 - n1 == (w["n_layers"] - 1) * _activation_set_bytes(w, B, S, fused)
    st, _ = _fake_workspace(lib, h, B, S, 0, None)
    assert st == 0 and _digest(lib, h) != d0
    m.set_recompute(False)
    assert m.workspace_bytes(B, S) == n0
    st, _ = _fake_workspace(lib, h, B, S, 0, None)
    assert st == 0 and _digest(lib, h) == d0


class _FakeTensor:
    """Stands in for a device tensor in the binding's operand checks (no memory behind it)."""

    def __init__(self, dtype, n, cuda=True, contiguous=True):
        import torch
        self.dtype = getattr(torch, dtype)
        self.is_cuda = cuda
        self._n = n
        self._c = contiguous

    def numel(self):
        return self._n

    def is_contiguous(self):
        return self._c

    def data_ptr(self):
        return 1 << 40


def test_binding_refuses_mismatched_operands_before_any_launch():
    pytest.importorskip("torch")
    m = _model("tiny-gpt2-fp32")
    P = m.num_params
    good = _FakeTensor("float32", P)
    tok = None
    cases = [
        (dict(params=_FakeTensor("bfloat16", P), v=good, out=good), "dtype"),
        (dict(params=good, v=_FakeTensor("float16", P), out=good), "dtype"),
        (dict(params=good, v=_FakeTensor("float32", P - 1), out=good), "elements"),
        (dict(params=good, v=good, out=_FakeTensor("float32", P, contiguous=False)), "contiguous"),
        (dict(params=good, v=_FakeTensor("float32", P, cuda=False), out=good), "device"),
        (dict(params=_FakeTensor("float32", 2 * P), v=good, out=good), "elements"),
    ]
    for kw, word in cases:
        with pytest.raises(ValueError, match=word):
            m.hvp(kw["params"], kw["v"], 1e-3, tok, out=kw["out"])
    with pytest.raises(ValueError):
        m.hvp_bound(_FakeTensor("float64", P), out=good)
    with pytest.raises(ValueError):
        m.block_stats(good, _FakeTensor("float32", P + 8))
    with pytest.raises(ValueError):
        m.cg_solve(_FakeTensor("int32", P), 1.0, 2, x=good)
    q = fd.Model("quad_diag", quad_n=1000)
    with pytest.raises(ValueError):
        q.set_quad_diag(_FakeTensor("float32", 999))
    bm = _model("llama-1.3b-bf16")
    with pytest.raises(ValueError, match="dtype"):
        bm.bind(_FakeTensor("float32", bm.num_params), None, 1e-3)


def test_block_stats_noalloc_refuses_too_many_blocks_before_any_launch():
    lib = fd.lib()
    cfg = fd.ModelConfig(1, 300, 8, 1, 1, 8, 8, 8, 0, 1e-5, 1e4, 0, 0)   # 300 tiny layers
    h = C.c_void_p()
    assert lib.fdh_create(C.byref(cfg), None, C.byref(h)) == 0
    out = np.zeros(3 * 300)
    st = lib.fdh_block_stats_noalloc(h, C.c_void_p(1 << 40), C.c_void_p(1 << 40),
                                     out.ctypes.data_as(C.POINTER(C.c_double)))
    assert st == -6 and b"256" in lib.fdh_last_error(h)
    assert lib.fdh_block_stats_noalloc(h, None, C.c_void_p(1 << 40), out.ctypes.data_as(C.POINTER(C.c_double))) == -1
    lib.fdh_destroy(h)
