"""Pins for the oracle's Lanczos / SLQ / block statistics (CPU, float64)."""
import numpy as np
import pytest

import synth
from oracle import block as B
from oracle import lanczos as L


def _diag_op(d):
    return lambda x: d * x


def test_diagonal_k_distinct_terminates_exactly():
    # k distinct eigenvalues => the Krylov space has dimension k: beta_{k+1} = 0,
    # Ritz values are the eigenvalues, weights the probe mass per eigenspace
    vals = np.array([-2.0, 0.5, 1.0, 3.0, 10.0])
    P = 1000
    d = vals[np.arange(P) % vals.size]
    q = synth.rademacher_probe(3, P).astype(np.float64)
    a, b, _ = L.lanczos(_diag_op(d), q, m=10, reorth=L.FULL)
    assert len(a) == vals.size
    assert b[-1] <= 1e-12 * np.abs(a).max()
    lam, tau = L.ritz(a, b)
    assert np.allclose(lam, vals, atol=1e-12)
    qn = q / np.linalg.norm(q)
    mass = np.array([np.sum(qn[d == x] ** 2) for x in vals])
    assert np.allclose(tau, mass, atol=1e-12)
    assert abs(tau.sum() - 1.0) < 1e-13


def test_full_dimension_reproduces_spectrum():
    rng = np.random.default_rng(0)
    P = 40
    A = rng.standard_normal((P, P))
    A = (A + A.T) / 2
    q = rng.standard_normal(P)
    a, b, Q = L.lanczos(lambda x: A @ x, q, m=P, reorth=L.FULL)
    assert len(a) == P
    lam, _ = L.ritz(a, b)
    assert np.allclose(lam, np.linalg.eigvalsh(A), atol=1e-10)
    Qm = np.stack(Q[:P])
    assert np.abs(Qm @ Qm.T - np.eye(P)).max() < 1e-12


def test_recurrence_and_moment_identities():
    rng = np.random.default_rng(1)
    P = 300
    A = rng.standard_normal((P, P))
    A = (A + A.T) / np.sqrt(P)
    q = rng.standard_normal(P)
    q /= np.linalg.norm(q)
    m = 8
    a, b, Q = L.lanczos(lambda x: A @ x, q, m=m, reorth=L.FULL)
    # alpha_1 = q^T H q ; alpha_1^2 + beta_2^2 = ||H q||^2
    assert abs(a[0] - q @ A @ q) < 1e-12
    assert abs(a[0] ** 2 + b[0] ** 2 - np.linalg.norm(A @ q) ** 2) < 1e-11
    # Gauss quadrature is exact for polynomials of degree <= 2m - 1
    lam, tau = L.ritz(a, b)
    x = q.copy()
    for j in range(2 * m):
        want = q @ x            # q^T A^j q
        got = np.sum(tau * lam ** j)
        assert abs(got - want) <= 1e-9 * max(1.0, abs(want)), j
        x = A @ x
    # three-term recurrence: A q_k = beta_k q_{k-1} + alpha_k q_k + beta_{k+1} q_{k+1}
    for k in range(1, m - 1):
        r = A @ Q[k] - b[k - 1] * Q[k - 1] - a[k] * Q[k] - b[k] * Q[k + 1]
        assert np.linalg.norm(r) < 1e-10


def test_slq_trace_diagonal_rademacher_exact():
    rng = np.random.default_rng(2)
    P = 500
    d = rng.standard_normal(P)
    probes = [synth.rademacher_probe(10 + j, P).astype(np.float64) for j in range(3)]
    nodes, weights, trace, steps = L.slq(_diag_op(d), probes, m=5)
    # z_i^2 = 1 => P * alpha_1 = z^T D z = tr(D) for every probe
    assert abs(trace - d.sum()) < 1e-9 * np.abs(d).sum()
    for w in weights:
        assert abs(w.sum() - 1.0) < 1e-12


def test_slq_trace_hutchinson_bound():
    rng = np.random.default_rng(3)
    P = 200
    A = rng.standard_normal((P, P))
    A = (A + A.T) / 2
    s = 64
    probes = [synth.rademacher_probe(100 + j, P).astype(np.float64) for j in range(s)]
    _, _, trace, _ = L.slq(lambda x: A @ x, probes, m=3)
    var = 2 * (np.linalg.norm(A) ** 2 - np.sum(np.diag(A) ** 2))
    assert abs(trace - np.trace(A)) <= 4 * np.sqrt(var / s)


def test_window_at_least_m_equals_full():
    rng = np.random.default_rng(4)
    P = 100
    A = rng.standard_normal((P, P))
    A = (A + A.T) / 2
    q = rng.standard_normal(P)
    a1, b1, _ = L.lanczos(lambda x: A @ x, q, m=12, reorth=L.FULL)
    a2, b2, _ = L.lanczos(lambda x: A @ x, q, m=12, reorth=L.WINDOW, window=12)
    assert np.array_equal(a1, a2) and np.array_equal(b1, b2)


@pytest.mark.parametrize("r", [1, 2, 4, 8])
def test_window_orthogonality_pattern(r):
    """Appendix C's window: the new Lanczos vector is reorthogonalised against
    the r most recent vectors (q_k among them).  Pinned by the orthogonality
    that leaves behind, on a spectrum with three outlying eigenvalues whose
    Ritz values converge within a few steps (so that plain Lanczos loses
    orthogonality quickly): every q_{k+1} is orthogonal to rounding level
    (1e-13) to each vector of its window, and its product with the vector just
    outside the window rises to far above that in some step (at least 1e-12
    and a thousand times the largest in-window product; the three-term
    recurrence itself keeps q_{k-1} close, so r = 1 shows the smallest gap).  A
    window one vector too wide passes the first test but fails the second; one
    too narrow fails the first."""
    P = 400
    d = np.concatenate([[100.0, 80.0, 60.0], np.linspace(-1, 1, P - 3)])
    q = np.random.default_rng(0).standard_normal(P)
    m = 60
    _, _, Q = L.lanczos(_diag_op(d), q, m, reorth=L.WINDOW, window=r)
    Q = np.array(Q)
    assert len(Q) == m + 1
    inside, outside = [], []
    for k in range(1, len(Q)):
        inside += [abs(Q[k] @ Q[j]) for j in range(max(0, k - r), k)]
        if k - r - 1 >= 0:
            outside.append(abs(Q[k] @ Q[k - r - 1]))
    assert max(inside) <= 1e-13
    assert max(outside) >= 1e-12 and max(outside) >= 1e3 * max(inside)
    # r = 1 and r = 2 keep only what the three-term recurrence already removes
    # in exact arithmetic: far older vectors lose orthogonality as without
    # reorthogonalisation
    assert max(abs(Q[k] @ Q[0]) for k in range(r + 1, len(Q))) >= 1e-6


def test_no_reorth_ghosts_appear():
    # section 4: without reorthogonalisation, converged Ritz values repeat ("ghosts")
    P = 400
    d = np.concatenate([[100.0], np.linspace(0, 1, P - 1)])
    q = np.ones(P) / np.sqrt(P)
    a, b, _ = L.lanczos(_diag_op(d), q, m=120, reorth=L.NONE)
    lam, _ = L.ritz(a, b)
    assert np.sum(np.abs(lam - 100.0) < 1e-6) >= 2
    a, b, _ = L.lanczos(_diag_op(d), q, m=120, reorth=L.FULL)
    lam, _ = L.ritz(a, b)
    assert np.sum(np.abs(lam - 100.0) < 1e-6) == 1


def test_block_stats_block_diagonal_operator():
    rng = np.random.default_rng(5)
    sizes = [30, 50, 20]
    Ab = []
    for n in sizes:
        M = rng.standard_normal((n, n))
        Ab.append(M + M.T)
    P = sum(sizes)
    A = np.zeros((P, P))
    blocks, off = [], 0
    for n, M in zip(sizes, Ab):
        A[off:off + n, off:off + n] = M
        blocks.append((off, off + n))
        off += n
    v = synth.gaussian_direction(4, P)
    st, h, hb = B.run(lambda x: A @ x, v, blocks)
    assert np.all(st["rel"] < 1e-12) and np.all(np.abs(st["cos"] - 1) < 1e-12)
    # a dense operator is not block diagonal
    A2 = A + 0.5 * rng.standard_normal((P, P))
    A2 = (A2 + A2.T) / 2
    st2, _, _ = B.run(lambda x: A2 @ x, v, blocks)
    assert st2["rel_mean"] > 0.1


def test_block_stats_formulas():
    h = np.array([1.0, 2.0, 3.0, 4.0])
    hb = [np.array([1.0, 0.0, 9, 9]), np.array([9, 9, 3.0, 0.0])]
    st = B.block_stats(h, hb, [(0, 2), (2, 4)])
    assert np.allclose(st["abs"], [2.0, 4.0])
    assert np.allclose(st["rel"], [2 / np.sqrt(5), 4 / 5])
    assert np.allclose(st["cos"], [1 / np.sqrt(5), 3 / 5])
    assert np.isclose(st["rel_std"], np.std([2 / np.sqrt(5), 4 / 5]))
