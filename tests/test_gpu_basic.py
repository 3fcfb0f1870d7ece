"""GPU checks of the building blocks through the C ABI: the MFMA GEMM, the
SplitMix64 input generators, and Lanczos / SLQ on the quadratic-diagonal
operator against the oracle."""
import numpy as np
import pytest

import synth
from oracle import lanczos as OL
from oracle import model as M
from synth.workloads import WORKLOADS
from tests import micro
from tests.gpu_util import need_gpu, say

pytestmark = pytest.mark.gpu


def _bf16_np(x):
    return synth.bf16_round(x.astype(np.float32))


@pytest.mark.parametrize("dtype,tile", [("bf16", 1), ("bf16", 2), ("bf16", 3), ("bf16", 4), ("bf16", 5), ("bf16", 6), ("bf16", 7), ("bf16", 8), ("f32", 0)])
@pytest.mark.parametrize("ak,bk", [(1, 1), (1, 0), (0, 1), (0, 0)])
def test_gemm_layouts_pairs_batches(dtype, tile, ak, bk):
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    say(f"gemm {dtype} tile={tile} ak={ak} bk={bk}")
    rng = np.random.default_rng(7)
    # ragged: several tiles and a tail in M, N and K for every tile variant
    # (the DMA-fed variants 4, 5 need K % 32 == 0)
    batch, M_, N_, K_ = (3, 200, 136, 72) if tile <= 1 else ((2, 296, 264, 200) if tile <= 3 else (2, 296, 264, 192))
    def mk(r, c):
        x = rng.standard_normal((batch, r, c)).astype(np.float32)
        return _bf16_np(x) if dtype == "bf16" else x
    A, B, A2, B2 = mk(M_, K_), mk(N_, K_), mk(M_, K_), mk(N_, K_)
    want = np.einsum("zmk,znk->zmn", A.astype(np.float64), B.astype(np.float64))
    want += np.einsum("zmk,znk->zmn", A2.astype(np.float64), B2.astype(np.float64))
    want *= 0.5
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    def up(x, kmaj):
        y = x if kmaj else np.ascontiguousarray(np.transpose(x, (0, 2, 1)))
        return torch.from_numpy(np.ascontiguousarray(y)).cuda().to(tdt)
    dA, dB, dA2, dB2 = up(A, ak), up(B, bk), up(A2, ak), up(B2, bk)
    C = torch.full((batch, M_, N_), float("nan"), device="cuda")
    fd.testing_gemm(dtype, M_, N_, K_, batch, ak, bk, dA, dB, dA2, dB2, C, 0, 0.5, tile)
    got = C.cpu().numpy().astype(np.float64)
    err = np.abs(got - want).max() / np.abs(want).max()
    assert err < 2e-6, err


@pytest.mark.parametrize("tile", [1, 2, 3, 4, 5, 6, 7, 8])
@pytest.mark.parametrize("causal", [1, 2, 3])
def test_gemm_causal_modes(causal, tile):
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    say(f"gemm causal {causal} tile {tile}")
    rng = np.random.default_rng(8)
    S = 320 if tile == 1 else (584 if tile <= 3 else 576)
    if causal == 1:     # scores: only tiles on/below the diagonal are produced
        M_, N_, K_ = S, S, 64
        A = _bf16_np(rng.standard_normal((2, M_, K_)))
        B = _bf16_np(rng.standard_normal((2, N_, K_)))
        ak = bk = 1
    else:               # contraction with a lower-triangular (2) or upper-triangular (3) A
        M_, N_, K_ = S, 64, S
        A = _bf16_np(rng.standard_normal((2, M_, K_)))
        tri = np.tril(np.ones((S, S))) if causal == 2 else np.triu(np.ones((S, S)))
        A = (A * tri).astype(np.float32)
        B = _bf16_np(rng.standard_normal((2, N_, K_)))
        ak = bk = 1
    want = np.einsum("zmk,znk->zmn", A.astype(np.float64), B.astype(np.float64))
    dA = torch.from_numpy(A).cuda().to(torch.bfloat16)
    dB = torch.from_numpy(B).cuda().to(torch.bfloat16)
    C = torch.zeros((2, M_, N_), device="cuda")
    fd.testing_gemm("bf16", M_, N_, K_, 2, ak, bk, dA, dB, None, None, C, causal, 1.0, tile)
    got = C.cpu().numpy().astype(np.float64)
    if causal == 1:
        i, j = np.tril_indices(S)
        err = np.abs(got[:, i, j] - want[:, i, j]).max() / np.abs(want).max()
    else:
        err = np.abs(got - want).max() / np.abs(want).max()
    assert err < 2e-6, err


@pytest.mark.parametrize("name", ["tiny-gpt2-fp32", "gpt2-medium-bf16", "llama3-8b-bf16"])
def test_init_params_matches_generator(name):
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    w = WORKLOADS[name]
    say(f"init params {name}")
    m = fd.Model.from_workload(w)
    p = m.init_params(1)
    torch.cuda.synchronize()
    cfg = micro.cfg_of(w)
    lay = M.layout(cfg)
    # compare the first 200k and last 200k entries and every non-matrix entry
    P = m.num_params
    idx = np.concatenate([np.arange(min(P, 200000)), np.arange(max(0, P - 200000), P)])
    ranges = [(e.offset, e.numel, e.kind) for e in lay]
    sub = synth.init_params(ranges, P, 1, bf16=w["dtype"] == "bf16") if P < 3e7 else None
    got = p.float().cpu().numpy() if P < 3e7 else p[torch.from_numpy(idx).cuda()].float().cpu().numpy()
    if sub is not None:
        want = sub
    else:
        want = np.zeros(idx.size, dtype=np.float32)
        for e in lay:
            sel = (idx >= e.offset) & (idx < e.offset + e.numel)
            if not sel.any():
                continue
            ii = idx[sel]
            if e.kind == M.MATRIX:
                vals = (0.02 * synth.normal(1, synth.STREAM_PARAMS, int(ii[0]), int(ii[-1] - ii[0] + 1))).astype(np.float32)
                want[sel] = vals[ii - ii[0]]
            else:
                want[sel] = 1.0 if e.kind == M.GAIN else 0.0
        if w["dtype"] == "bf16":
            want = synth.bf16_round(want)
    diff = np.abs(got.astype(np.float64) - want.astype(np.float64))
    ulp = np.spacing(np.abs(want).astype(np.float32)).astype(np.float64)
    if w["dtype"] == "bf16":
        ulp = ulp * 65536
    assert np.all(diff <= ulp), diff.max()
    assert (diff > 0).mean() < 1e-4


@pytest.mark.parametrize("dist", ["uniform", "zipf"])
def test_tokens_match_generator_bitwise(dist):
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    w = WORKLOADS["llama-1.3b-bf16"]
    m = fd.Model.from_workload(w)
    m.set_workspace(0, 0)
    t = m.make_tokens(4, 2048, 2, dist)
    torch.cuda.synchronize()
    want = synth.tokens(2, 4, 2048, w["vocab"], dist)
    assert np.array_equal(t.cpu().numpy(), want)


def test_probe_vectors_match_generator():
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    m = fd.Model("quad_diag", quad_n=100003)
    m.set_workspace()
    r = m.random_vector(5, "rademacher").cpu().numpy()
    assert np.array_equal(r, synth.rademacher_probe(5, 100003))
    g = m.random_vector(6, "gaussian").cpu().numpy().astype(np.float64)
    want = synth.gaussian_direction(6, 100003)
    assert np.abs(g - want).max() < 1e-7


def _quad_setup(torch, fd, diag, m_steps, reorth="full", window=0, basis="f32"):
    P = diag.size
    mod = fd.Model("quad_diag", quad_n=P)
    o = fd.opts(reorth, window, basis)
    mod.set_workspace(0, 0, m_steps, o)
    d = torch.from_numpy(diag.astype(np.float32)).cuda()
    th = torch.from_numpy(np.linspace(-1, 1, P).astype(np.float32)).cuda()
    mod.set_quad_diag(d)
    mod.bind(th, None, 1e-3)
    mod._keep += [d, th]
    return mod, o, th


def test_quad_diag_hvp_exact():
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    P = 50001
    rng = np.random.default_rng(1)
    diag = rng.standard_normal(P).astype(np.float32)
    mod, _, th = _quad_setup(torch, fd, diag, 1)
    v = torch.from_numpy(synth.gaussian_direction(3, P).astype(np.float32)).cuda()
    hv = mod.hvp(th, v, 1e-3).cpu().numpy().astype(np.float64)
    want = diag.astype(np.float64) * v.cpu().numpy().astype(np.float64)
    assert np.abs(hv - want).max() <= 1e-6 * np.abs(want).max()


def test_lanczos_quad_diag_distinct_eigenvalues():
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    vals = np.array([-2.0, 0.5, 1.0, 3.0, 10.0])
    P = 100000
    diag = vals[np.arange(P) % vals.size]
    mod, o, _ = _quad_setup(torch, fd, diag, 10)
    a, b, s, st = mod.lanczos(10, 3, o)
    assert st == fd.BREAKDOWN and s == 5
    lam = np.sort(np.linalg.eigvalsh(OL.tridiag(a[:s], b[:s])))
    assert np.allclose(lam, vals, atol=1e-4)


@pytest.mark.parametrize("reorth,window,basis", [("full", 0, "f32"), ("full", 0, "bf16"), ("window", 4, "f32"), ("none", 0, "f32")])
def test_lanczos_quad_diag_matches_oracle(reorth, window, basis):
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    say(f"lanczos quad {reorth} {window} {basis}")
    P = 200003
    rng = np.random.default_rng(2)
    diag = np.concatenate([[50.0, 40.0, -30.0], rng.uniform(-1, 1, P - 3)]).astype(np.float32)
    m = 16
    mod, o, _ = _quad_setup(torch, fd, diag, m, reorth, window, basis)
    a, b, s, st = mod.lanczos(m, 11, o)
    assert s == m and st == fd.OK
    q1 = synth.rademacher_probe(11, P).astype(np.float64)
    ro = {"full": OL.FULL, "window": OL.WINDOW, "none": OL.NONE}[reorth]
    ao, bo, _ = OL.lanczos(lambda x: diag.astype(np.float64) * x, q1, m, ro, window)
    lam_g = np.sort(np.linalg.eigvalsh(OL.tridiag(a, b)))
    lam_o = np.sort(np.linalg.eigvalsh(OL.tridiag(ao, bo)))
    scale = np.abs(lam_o).max()
    say(f"  extreme Ritz errors {abs(lam_g[-1] - lam_o[-1]) / scale:.3e}, {abs(lam_g[0] - lam_o[0]) / scale:.3e}; "
        f"alpha_1 {abs(a[0] - ao[0]) / scale:.3e}")
    # extreme Ritz values within 1e-3 relative (fp32).  A bf16 basis stores every
    # row with a relative rounding of at most 2^-9, so the reorthogonalisation
    # removes the stored directions only to that accuracy and the Ritz values
    # of the perturbed recurrence move by about 2^-9 of the spectral scale at
    # first order: the bar is 2^-8 (measured 1.0e-4 and 8.8e-4 at m = 16)
    tol = 1e-3 if basis == "f32" else 2.0 ** -8
    assert abs(lam_g[-1] - lam_o[-1]) <= tol * scale
    assert abs(lam_g[0] - lam_o[0]) <= tol * scale
    assert abs(a[0] - ao[0]) <= 1e-5 * scale


@pytest.mark.parametrize("m,basis", [(24, "f32"), (40, "bf16"), (72, "f32"), (100, "bf16")])
def test_lanczos_long_runs_match_oracle(m, basis):
    """Full reorthogonalisation with up to 100 stored rows (every row-group
    width of the projection kernel) on a length that is not a multiple of 8."""
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    say(f"lanczos long run m={m} {basis}")
    P = 50003
    rng = np.random.default_rng(4)
    diag = np.concatenate([np.linspace(-5.0, 100.0, 40), rng.uniform(-1, 1, P - 40)]).astype(np.float32)
    mod, o, _ = _quad_setup(torch, fd, diag, m, "full", 0, basis)
    a, b, s, st = mod.lanczos(m, 5, o)
    assert s == m and st == fd.OK
    q1 = synth.rademacher_probe(5, P).astype(np.float64)
    ao, bo, _ = OL.lanczos(lambda x: diag.astype(np.float64) * x, q1, m, OL.FULL, 0)
    lam_g = np.sort(np.linalg.eigvalsh(OL.tridiag(a, b)))
    lam_o = np.sort(np.linalg.eigvalsh(OL.tridiag(ao, bo)))
    scale = np.abs(lam_o).max()
    # the five largest of this spectrum are well separated and converged after
    # 24 steps, which damps the basis rounding well below its 2^-9 first-order
    # size: 5e-4 holds for the bf16 basis here
    tol = 1e-5 if basis == "f32" else 5e-4
    assert np.abs(lam_g[-5:] - lam_o[-5:]).max() <= tol * scale
    assert abs(lam_g[0] - lam_o[0]) <= tol * scale


def test_slq_quad_diag_trace_and_weights():
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    P = 100000
    rng = np.random.default_rng(3)
    diag = rng.standard_normal(P).astype(np.float32)
    mod, o, _ = _quad_setup(torch, fd, diag, 8)
    nodes, weights, steps, trace, st = mod.slq_density(3, 8, 20, o)
    # Rademacher probes: P * alpha_1 = tr(D) exactly for a diagonal operator
    assert abs(trace - diag.astype(np.float64).sum()) <= 1e-4 * np.abs(diag).sum()
    assert np.allclose(weights.sum(1), 1.0, atol=1e-9)
    probes = [synth.rademacher_probe(20 + j, P).astype(np.float64) for j in range(3)]
    no, wo, tro, _ = OL.slq(lambda x: diag.astype(np.float64) * x, probes, 8)
    for j in range(3):
        assert np.abs(nodes[j] - no[j]).max() <= 1e-4 * np.abs(no[j]).max()
        assert np.abs(weights[j] - wo[j]).max() <= 1e-4
