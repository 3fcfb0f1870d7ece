"""Python binding of libfdhvp (include/fdhvp.h): argument marshalling only.

Every computation runs in the HIP library; PyTorch supplies device memory and
the current stream.  Loading fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libfdhvp.so")

# enums (include/fdhvp.h)
OK, BREAKDOWN = 0, 1
ERR = {-1: "INVALID_ARG", -2: "WORKSPACE", -3: "HIP", -4: "NONFINITE", -5: "STATE", -6: "UNSUPPORTED"}
FAMILY = {"gpt2": 0, "llama": 1, "quad_diag": 2}
DTYPE = {"f32": 0, "bf16": 1}
REORTH = {"none": 0, "full": 1, "window": 2}
TOKENS = {"uniform": 0, "zipf": 1}
VEC = {"rademacher": 0, "gaussian": 1}
REDUCTION = {"mean": 0, "sum": 1}
IGNORE = -100


class FdhError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"fdhvp error {ERR.get(status, status)}: {msg}")
        self.status = status


class ModelConfig(C.Structure):
    _fields_ = [("family", C.c_int32), ("n_layers", C.c_int32), ("d_model", C.c_int32),
                ("n_heads", C.c_int32), ("n_kv_heads", C.c_int32), ("d_ff", C.c_int32),
                ("vocab", C.c_int32), ("max_seq", C.c_int32), ("dtype", C.c_int32),
                ("norm_eps", C.c_float), ("rope_base", C.c_float), ("reserved", C.c_int32),
                ("quad_n", C.c_int64)]


class LanczosOpts(C.Structure):
    _fields_ = [("reorth", C.c_int32), ("window", C.c_int32), ("basis_dtype", C.c_int32),
                ("breakdown_tol", C.c_float)]


class Batch(C.Structure):
    _fields_ = [("tokens", C.c_void_p), ("labels", C.c_void_p), ("B", C.c_int32), ("S", C.c_int32)]


class Block(C.Structure):
    _fields_ = [("name", C.c_char * 48), ("offset", C.c_int64), ("numel", C.c_int64),
                ("rows", C.c_int64), ("cols", C.c_int64), ("layer", C.c_int32), ("kind", C.c_int32)]


_lib = None


def lib():
    """The loaded shared library (raises if it is missing)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2602_00816_amd.build`")
    L = C.CDLL(LIB_PATH)
    vp, i32, i64, u64, f64 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64, C.c_double
    pd, pi = C.POINTER(C.c_double), C.POINTER(C.c_int32)
    sig = {
        "fdh_api_version": (i32, []),
        "fdh_create": (i32, [C.POINTER(ModelConfig), vp, C.POINTER(vp)]),
        "fdh_destroy": (None, [vp]),
        "fdh_num_params": (i64, [vp]),
        "fdh_num_blocks": (i32, [vp]),
        "fdh_param_layout": (i32, [vp, C.POINTER(Block), i32, pi]),
        "fdh_workspace_bytes": (i32, [vp, i32, i32, i32, C.POINTER(LanczosOpts), C.POINTER(C.c_size_t)]),
        "fdh_set_workspace": (i32, [vp, vp, C.c_size_t, i32, i32, i32, C.POINTER(LanczosOpts)]),
        "fdh_set_recompute": (i32, [vp, i32]),
        "fdh_init_params": (i32, [vp, vp, u64]),
        "fdh_make_tokens": (i32, [vp, vp, i32, i32, u64, i32]),
        "fdh_random_vector": (i32, [vp, vp, u64, i32]),
        "fdh_set_quad_diag": (i32, [vp, vp]),
        "fdh_hvp": (i32, [vp, vp, vp, f64, vp, i32, i32, vp]),
        "fdh_last_losses": (i32, [vp, pd, pd]),
        "fdh_bind": (i32, [vp, vp, vp, i32, i32, f64]),
        "fdh_bind_dataset": (i32, [vp, vp, C.POINTER(Batch), i32, f64, i32, C.POINTER(i64)]),
        "fdh_hvp_bound": (i32, [vp, vp, vp]),
        "fdh_set_basis_offload": (i32, [vp, i32, vp, C.c_size_t]),
        "fdh_lanczos": (i32, [vp, i32, u64, C.POINTER(LanczosOpts), pd, pd, pi]),
        "fdh_slq_density": (i32, [vp, i32, i32, u64, C.POINTER(LanczosOpts), pd, pd, pi, pd]),
        "fdh_block_stats": (i32, [vp, vp, vp, pd]),
        "fdh_block_stats_noalloc": (i32, [vp, vp, vp, pd]),
        "fdh_block_diagonal": (i32, [vp, vp, pd]),
        "fdh_cg_solve": (i32, [vp, vp, C.c_double, i32, C.c_double, vp, pd, C.POINTER(C.c_int32)]),
        "fdh_last_error": (C.c_char_p, [vp]),
        "fdh_ritz_diagnostics": (i32, [pd, pd, i32, f64, pd, pd, pd, pi, pi, pi]),
        "fdh_testing_gemm": (i32, [i32, i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp, i32, C.c_float, i32, vp]),
        "fdh_testing_gemm_pair": (i32, [i32, i32, i32, i32, i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp,
                                        vp, vp, C.c_float, i32, vp]),
        "fdh_testing_unfused_attention": (i32, [vp, i32]),
        "fdh_testing_unsplit_wgrad": (i32, [vp, i32]),
        "fdh_testing_timing": (i32, [vp, i32]),
        "fdh_testing_timing_read": (i32, [vp, pd]),
        "fdh_testing_copy": (i32, [vp, vp, C.c_size_t, vp]),
        "fdh_testing_layout_digest": (i32, [vp, C.POINTER(C.c_uint64)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _check_tokens(t):
    import torch
    if t is not None and (t.dtype != torch.int32 or t.dim() != 2 or not t.is_cuda or not t.is_contiguous()):
        raise ValueError("tokens must be a contiguous int32 [B, S] tensor on the device")


def _check_vec(t, n: int, what: str, dtypes=("float32",), optional=False):
    """A parameter-sized device operand: the kernels read or write exactly n
    elements of the given type through its pointer, so anything else (another
    dtype, a short or strided tensor, host memory) is refused here, before any
    launch."""
    if t is None:
        if optional:
            return
        raise ValueError(f"{what} is required")
    if not hasattr(t, "data_ptr") or not hasattr(t, "is_cuda"):
        raise ValueError(f"{what} must be a torch tensor on the device")
    dt = str(t.dtype).replace("torch.", "")
    if dt not in dtypes:
        raise ValueError(f"{what} must have dtype {' or '.join(dtypes)}, not {dt}")
    if not t.is_cuda:
        raise ValueError(f"{what} must be on the device")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if t.numel() != n:
        raise ValueError(f"{what} must have {n} elements, not {t.numel()}")


def _stream():
    import torch
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def opts(reorth="full", window=0, basis="f32", tol=0.0) -> LanczosOpts:
    return LanczosOpts(REORTH[reorth], int(window), DTYPE[basis], float(tol))


@dataclass
class Entry:
    name: str
    offset: int
    numel: int
    rows: int
    cols: int
    layer: int
    kind: int


class Model:
    """One fdh_ctx: a model (or the quadratic test operator) on the current GPU."""

    def __init__(self, family: str, n_layers=0, d_model=0, n_heads=1, n_kv_heads=0, d_ff=0, vocab=0,
                 max_seq=0, dtype="f32", norm_eps=1e-5, rope_base=10000.0, quad_n=0, stream=None):
        self._L = lib()
        self.cfg = ModelConfig(FAMILY[family], n_layers, d_model, n_heads, n_kv_heads or n_heads, d_ff, vocab,
                               max_seq, DTYPE[dtype], norm_eps, rope_base, 0, quad_n)
        self.family, self.dtype = family, dtype
        h = C.c_void_p()
        st = self._L.fdh_create(C.byref(self.cfg), stream if stream is not None else C.c_void_p(0), C.byref(h))
        if st != OK:
            raise FdhError(st, "fdh_create rejected the configuration")
        self._h = h
        self._ws = None
        self._keep = []        # tensors the bound operator points to
        self._diag = None      # QUAD_DIAG diagonal the context points to

    @classmethod
    def from_workload(cls, w: dict, stream=None):
        return cls(w["family"], w["n_layers"], w["d_model"], w["n_heads"], w["n_kv_heads"], w["d_ff"],
                   w["vocab"], w["max_seq"], w["dtype"], rope_base=w["rope_base"], stream=stream)

    def close(self):
        if getattr(self, "_h", None):
            self._L.fdh_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _param_dtypes(self):
        return ("float32",) if self.dtype == "f32" else ("bfloat16", "uint16", "int16")

    def _check_params(self, p):
        _check_vec(p, self.num_params, "params", self._param_dtypes())

    def _check_vec(self, t, what, optional=False):
        _check_vec(t, self.num_params, what, optional=optional)

    def _check(self, st: int, what: str) -> int:
        if st < 0:
            msg = self._L.fdh_last_error(self._h)
            raise FdhError(st, f"{what}: {msg.decode() if msg else ''}")
        return st

    # ---- description ----
    @property
    def num_params(self) -> int:
        return int(self._L.fdh_num_params(self._h))

    @property
    def num_blocks(self) -> int:
        return int(self._L.fdh_num_blocks(self._h))

    def layout(self) -> list[Entry]:
        n = C.c_int32()
        self._check(self._L.fdh_param_layout(self._h, None, 0, C.byref(n)), "fdh_param_layout")
        arr = (Block * n.value)()
        self._check(self._L.fdh_param_layout(self._h, arr, n.value, C.byref(n)), "fdh_param_layout")
        return [Entry(b.name.decode(), b.offset, b.numel, b.rows, b.cols, b.layer, b.kind) for b in arr]

    def workspace_bytes(self, B=0, S=0, m=0, o: LanczosOpts | None = None) -> int:
        out = C.c_size_t()
        self._check(self._L.fdh_workspace_bytes(self._h, B, S, m, C.byref(o) if o else None, C.byref(out)),
                    "fdh_workspace_bytes")
        return int(out.value)

    def set_recompute(self, on: bool = True):
        """Activation recomputation for the following workspace_bytes /
        set_workspace: keep only each layer's input pair and rerun the layer's
        forward before its backward (same results, less memory)."""
        self._check(self._L.fdh_set_recompute(self._h, 1 if on else 0), "fdh_set_recompute")

    # ---- memory ----
    def set_workspace(self, B=0, S=0, m=0, o: LanczosOpts | None = None):
        import torch
        n = self.workspace_bytes(B, S, m, o)
        # detach before the old buffer goes back to torch, so that the context
        # never points at freed memory (also when the new size is refused)
        self._check(self._L.fdh_set_workspace(self._h, None, 0, 0, 0, 0, None), "fdh_set_workspace")
        self._ws = None
        buf = torch.empty(max(n, 256) + 256, dtype=torch.uint8, device="cuda")
        base = buf.data_ptr()
        off = (-base) % 256
        self._ws = buf
        self._check(self._L.fdh_set_workspace(self._h, C.c_void_p(base + off), n, B, S, m,
                                              C.byref(o) if o else None), "fdh_set_workspace")
        return n

    def empty_params(self):
        import torch
        dt = torch.float32 if self.dtype == "f32" else torch.uint16 if hasattr(torch, "uint16") else torch.int16
        if self.dtype == "bf16":
            dt = torch.bfloat16
        return torch.empty(self.num_params, dtype=dt, device="cuda")

    def init_params(self, seed: int):
        p = self.empty_params()
        self._check_params(p)
        self._check(self._L.fdh_init_params(self._h, _ptr(p), seed), "fdh_init_params")
        return p

    def make_tokens(self, B: int, S: int, seed: int, dist="uniform"):
        import torch
        t = torch.empty((B, S), dtype=torch.int32, device="cuda")
        self._check(self._L.fdh_make_tokens(self._h, _ptr(t), B, S, seed, TOKENS[dist]), "fdh_make_tokens")
        return t

    def random_vector(self, seed: int, kind="rademacher", out=None):
        import torch
        v = torch.empty(self.num_params, dtype=torch.float32, device="cuda") if out is None else out
        self._check_vec(v, "out")
        self._check(self._L.fdh_random_vector(self._h, _ptr(v), seed, VEC[kind]), "fdh_random_vector")
        return v

    def set_quad_diag(self, diag):
        self._check_vec(diag, "diag")
        self._diag = diag
        self._check(self._L.fdh_set_quad_diag(self._h, _ptr(diag)), "fdh_set_quad_diag")

    # ---- the hot path ----
    def hvp(self, params, v, eps: float, tokens=None, out=None):
        """Hv (float32 [P]) of the FD-HVP at step eps; enqueued on the context stream."""
        import torch
        if out is None:
            out = torch.empty(self.num_params, dtype=torch.float32, device="cuda")
        self._check_params(params)
        self._check_vec(v, "v")
        self._check_vec(out, "out")
        _check_tokens(tokens)
        B, S = (tokens.shape if tokens is not None else (0, 0))
        self._check(self._L.fdh_hvp(self._h, _ptr(params), _ptr(v), float(eps), _ptr(tokens), B, S, _ptr(out)),
                    "fdh_hvp")
        return out

    def last_losses(self):
        lp, lm = C.c_double(), C.c_double()
        self._check(self._L.fdh_last_losses(self._h, C.byref(lp), C.byref(lm)), "fdh_last_losses")
        return lp.value, lm.value

    def bind(self, params, tokens, eps: float):
        self._check_params(params)
        _check_tokens(tokens)
        B, S = (tokens.shape if tokens is not None else (0, 0))
        self._keep = [params, tokens]
        self._check(self._L.fdh_bind(self._h, _ptr(params), _ptr(tokens), B, S, float(eps)), "fdh_bind")

    def bind_dataset(self, params, batches, eps: float, reduction: str = "mean") -> int:
        """Bind the token-weighted dataset operator over ``batches``: a list of
        int32 [B, S] token tensors or (tokens, labels) pairs on the device
        (labels aligned with the tokens, -100 = no target).  Returns the number
        of kept targets."""
        import torch
        self._check_params(params)
        items = [b if isinstance(b, tuple) else (b, None) for b in batches]
        for tok, lab in items:
            for x in (tok, lab):
                if x is not None and (x.dtype != torch.int32 or x.dim() != 2 or not x.is_cuda or not x.is_contiguous()):
                    raise ValueError("tokens and labels must be contiguous int32 [B, S] tensors on the device")
            if lab is not None and lab.shape != tok.shape:
                raise ValueError("labels must have the shape of their tokens")
        arr = (Batch * len(items))(*[Batch(_ptr(t), _ptr(l), t.shape[0], t.shape[1]) for t, l in items])
        n = C.c_int64()
        self._keep = [params] + [x for it in items for x in it if x is not None]
        self._check(self._L.fdh_bind_dataset(self._h, _ptr(params), arr, len(items), float(eps), REDUCTION[reduction],
                                             C.byref(n)), "fdh_bind_dataset")
        return int(n.value)

    def hvp_bound(self, v, out=None):
        """H v of the bound operator (float32 [P]); enqueued on the context stream."""
        import torch
        if out is None:
            out = torch.empty(self.num_params, dtype=torch.float32, device="cuda")
        self._check_vec(v, "v")
        self._check_vec(out, "out")
        self._check(self._L.fdh_hvp_bound(self._h, _ptr(v), _ptr(out)), "fdh_hvp_bound")
        return out

    def set_basis_offload(self, device_rows: int, host_rows=None):
        """Keep at most device_rows Lanczos rows on the device and the rest in
        host_rows (a pinned host tensor, e.g. torch.empty(n, dtype=torch.uint8,
        pin_memory=True)); device_rows < 0 undoes it.  Call before set_workspace."""
        self._host_rows = host_rows
        nbytes = 0 if host_rows is None else host_rows.numel() * host_rows.element_size()
        self._check(self._L.fdh_set_basis_offload(self._h, int(device_rows), _ptr(host_rows), nbytes),
                    "fdh_set_basis_offload")

    def lanczos(self, m: int, probe_seed: int, o: LanczosOpts):
        a = np.zeros(m)
        b = np.zeros(m)
        s = C.c_int32()
        st = self._check(self._L.fdh_lanczos(self._h, m, probe_seed, C.byref(o),
                                             a.ctypes.data_as(C.POINTER(C.c_double)),
                                             b.ctypes.data_as(C.POINTER(C.c_double)), C.byref(s)), "fdh_lanczos")
        return a, b, int(s.value), st

    def slq_density(self, probes: int, m: int, seed: int, o: LanczosOpts):
        nodes = np.zeros((probes, m))
        weights = np.zeros((probes, m))
        steps = np.zeros(probes, dtype=np.int32)
        tr = C.c_double()
        st = self._check(self._L.fdh_slq_density(
            self._h, probes, m, seed, C.byref(o), nodes.ctypes.data_as(C.POINTER(C.c_double)),
            weights.ctypes.data_as(C.POINTER(C.c_double)), steps.ctypes.data_as(C.POINTER(C.c_int32)),
            C.byref(tr)), "fdh_slq_density")
        return nodes, weights, steps, tr.value, st

    def cg_solve(self, b, lam: float, max_iters: int, rel_tol: float = 0.0, x=None):
        """CG for (H + lam I) x = b on the bound operator (b: float32 [P] on device).
        Returns (x, residual norms ||r_0|| .. ||r_s||, s, status)."""
        import torch
        self._check_vec(b, "b")
        if x is None:
            x = torch.empty_like(b)
        self._check_vec(x, "x")
        res = np.zeros(max_iters + 1)
        s = C.c_int32()
        st = self._check(self._L.fdh_cg_solve(self._h, _ptr(b), float(lam), int(max_iters), float(rel_tol), _ptr(x),
                                              res.ctypes.data_as(C.POINTER(C.c_double)), C.byref(s)), "fdh_cg_solve")
        return x, res[:int(s.value) + 1], int(s.value), st

    def unfused_attention(self, on: bool):
        """Plan the unfused attention path at the next set_workspace (testing)."""
        self._check(self._L.fdh_testing_unfused_attention(self._h, int(on)), "fdh_testing_unfused_attention")

    def unsplit_wgrad(self, on):
        """Weight-gradient launch form (testing): False/0 default (token slices,
        shared launches), True/1 one launch over all tokens per weight, 2 token
        slices without shared launches."""
        self._check(self._L.fdh_testing_unsplit_wgrad(self._h, int(on)), "fdh_testing_unsplit_wgrad")

    def layout_digest(self) -> int:
        """Digest of the workspace carve in use (testing; host only)."""
        out = C.c_uint64()
        self._check(self._L.fdh_testing_layout_digest(self._h, C.byref(out)), "fdh_testing_layout_digest")
        return int(out.value)

    def timing(self, enable: bool):
        self._check(self._L.fdh_testing_timing(self._h, int(enable)), "fdh_testing_timing")

    def timing_read(self) -> dict:
        out = np.zeros(16)
        self._check(self._L.fdh_testing_timing_read(self._h, out.ctypes.data_as(C.POINTER(C.c_double))),
                    "fdh_testing_timing_read")
        cats = ["gemm", "lanczos", "attention", "c3"]
        return {c: dict(launches=out[4 * i], ms=out[4 * i + 1], flops=out[4 * i + 2], bytes=out[4 * i + 3])
                for i, c in enumerate(cats)}

    def block_diagonal(self, v):
        """Exp I statistics per layer: columns abs diff, relative error, cosine, ||(Hv)^(b)||."""
        self._check_vec(v, "v")
        out = np.zeros((max(self.num_blocks, 0), 4))
        self._check(self._L.fdh_block_diagonal(self._h, _ptr(v), out.ctypes.data_as(C.POINTER(C.c_double))),
                    "fdh_block_diagonal")
        return out

    def block_stats_noalloc(self, a, b):
        """fdh_block_stats without the workspace (fixed device scratch; no allocation)."""
        self._check_vec(a, "a")
        self._check_vec(b, "b")
        out = np.zeros((max(self.num_blocks, 0), 3))
        self._check(self._L.fdh_block_stats_noalloc(self._h, _ptr(a), _ptr(b),
                                                    out.ctypes.data_as(C.POINTER(C.c_double))),
                    "fdh_block_stats_noalloc")
        return out

    def block_stats(self, a, b):
        self._check_vec(a, "a")
        self._check_vec(b, "b")
        out = np.zeros((max(self.num_blocks, 0), 3))
        self._check(self._L.fdh_block_stats(self._h, _ptr(a), _ptr(b), out.ctypes.data_as(C.POINTER(C.c_double))),
                    "fdh_block_stats")
        return out


def ritz_diagnostics(alpha, beta, tol: float = 1e-8):
    """Ritz-value diagnostics of T_s (include/fdhvp.h: fdh_ritz_diagnostics).
    Returns (nodes, weights, resid, copies, spurious, n_ghosts)."""
    a = np.ascontiguousarray(alpha, dtype=np.float64)
    b = np.ascontiguousarray(beta, dtype=np.float64)
    s = a.size
    if b.size < s:
        raise ValueError("beta needs as many entries as alpha")
    nodes, weights, resid = np.zeros(s), np.zeros(s), np.zeros(s)
    copies, spurious, ng = np.zeros(s, np.int32), np.zeros(s, np.int32), C.c_int32()
    dp = lambda x: x.ctypes.data_as(C.POINTER(C.c_double))
    ip = lambda x: x.ctypes.data_as(C.POINTER(C.c_int32))
    st = lib().fdh_ritz_diagnostics(dp(a), dp(b), s, float(tol), dp(nodes), dp(weights), dp(resid), ip(copies),
                                    ip(spurious), C.byref(ng))
    if st != OK:
        raise FdhError(st, "fdh_ritz_diagnostics")
    return nodes, weights, resid, copies, spurious.astype(bool), int(ng.value)


def testing_copy(dst, src, nbytes: int):
    st = lib().fdh_testing_copy(_ptr(dst), _ptr(src), int(nbytes), _stream())
    if st != OK:
        raise FdhError(st, "fdh_testing_copy")


def testing_gemm(dtype: str, M, N, K, batch, a_kmajor, b_kmajor, A, B, A2, B2, Cout, causal=0, alpha=1.0, tile=0):
    st = lib().fdh_testing_gemm(DTYPE[dtype], M, N, K, batch, int(a_kmajor), int(b_kmajor), _ptr(A), _ptr(B),
                                _ptr(A2), _ptr(B2), _ptr(Cout), causal, float(alpha), int(tile), _stream())
    if st != OK:
        raise FdhError(st, "fdh_testing_gemm")


def testing_gemm_pair(M0, N0, K0, M1, N1, K1, a_kmajor, b_kmajor, P0, P1, alpha=1.0, tile=6, batch0=1, batch1=1):
    """Two bf16 products in one launch (testing); P_q = (A, B, A2, B2, C), A2/B2 may be None."""
    import torch
    A0, B0, A20, B20, C0 = P0
    A1, B1, A21, B21, C1 = P1
    for (M, N, K, z, (A, B, A2, B2, Cq)) in ((M0, N0, K0, batch0, P0), (M1, N1, K1, batch1, P1)):
        for t, n, dt in ((A, z * M * K, torch.bfloat16), (B, z * N * K, torch.bfloat16), (A2, z * M * K, torch.bfloat16),
                         (B2, z * N * K, torch.bfloat16), (Cq, z * M * N, torch.float32)):
            if t is not None and (not t.is_cuda or not t.is_contiguous() or t.dtype != dt or t.numel() != n):
                raise ValueError("testing_gemm_pair: operand of the wrong device, layout, type or size")
    st = lib().fdh_testing_gemm_pair(M0, N0, K0, int(batch0), M1, N1, K1, int(batch1), int(a_kmajor), int(b_kmajor),
                                     _ptr(A0), _ptr(B0),
                                     _ptr(A20), _ptr(B20), _ptr(C0), _ptr(A1), _ptr(B1), _ptr(A21), _ptr(B21),
                                     _ptr(C1), float(alpha), int(tile), _stream())
    if st != OK:
        raise FdhError(st, "fdh_testing_gemm_pair")
