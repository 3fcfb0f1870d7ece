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
