"""The CG oracle pinned to linear algebra it must reproduce (CPU only).

* On a random symmetric positive definite system it reaches np.linalg.solve.
* With exact arithmetic CG terminates in at most k steps when A has k distinct
  eigenvalues (Hestenes-Stiefel); in fp64 on a well-conditioned spectrum the
  residual after k steps is at rounding level, and not before.
* The damping enters as A = H + lam I: the solution of the shifted system.
* The residual norms it reports are those of b - A x_k, recomputed here.
* A direction of non-positive curvature stops it with the breakdown status.
"""
import numpy as np

from oracle import cg as OC


def _spd(n, seed, lo=0.5, hi=5.0):
    rng = np.random.default_rng(seed)
    q, _ = np.linalg.qr(rng.standard_normal((n, n)))
    ev = rng.uniform(lo, hi, n)
    return (q * ev) @ q.T


def test_cg_solves_spd_system():
    A = _spd(60, 1)
    b = np.random.default_rng(2).standard_normal(60)
    x, steps, res, st = OC.cg(lambda v: A @ v, b, 0.0, 200, 1e-13)
    assert st == OC.OK
    assert np.allclose(x, np.linalg.solve(A, b), rtol=1e-9, atol=1e-11)
    assert res[-1] <= 1e-13 * np.linalg.norm(b)


def test_cg_finite_termination_on_k_distinct_eigenvalues():
    n, k = 200, 5
    rng = np.random.default_rng(3)
    q, _ = np.linalg.qr(rng.standard_normal((n, n)))
    ev = np.array([1.0, 2.0, 3.5, 5.0, 8.0])[rng.integers(0, k, n)]
    A = (q * ev) @ q.T
    b = rng.standard_normal(n)
    x, steps, res, st = OC.cg(lambda v: A @ v, b, 0.0, k, 0.0)
    assert steps == k
    assert res[-1] <= 1e-10 * np.linalg.norm(b)
    assert res[k - 1] > 1e-6 * np.linalg.norm(b)   # not yet converged one step earlier
    assert np.allclose(x, np.linalg.solve(A, b), rtol=1e-8, atol=1e-10)


def test_cg_damping_shifts_the_operator():
    H = _spd(40, 4, lo=-1.0, hi=3.0)              # indefinite
    lam = 1.5                                      # H + lam I is positive definite
    b = np.random.default_rng(5).standard_normal(40)
    x, steps, res, st = OC.cg(lambda v: H @ v, b, lam, 200, 1e-13)
    assert st == OC.OK
    assert np.allclose(x, np.linalg.solve(H + lam * np.eye(40), b), rtol=1e-8, atol=1e-10)


def test_cg_reported_residuals_are_true_residuals():
    A = _spd(30, 6)
    b = np.random.default_rng(7).standard_normal(30)
    for m in range(1, 8):
        x, steps, res, st = OC.cg(lambda v: A @ v, b, 0.0, m, 0.0)
        assert steps == m
        assert abs(res[-1] - np.linalg.norm(b - A @ x)) <= 1e-10 * np.linalg.norm(b)
    assert np.all(np.diff(res) != 0.0)


def test_cg_breakdown_on_negative_curvature():
    A = np.diag([-1.0, 2.0, 3.0])
    b = np.array([1.0, 0.0, 0.0])                  # b is an eigenvector of eigenvalue -1
    x, steps, res, st = OC.cg(lambda v: A @ v, b, 0.0, 5, 0.0)
    assert st == OC.BREAKDOWN and steps == 0
    assert np.array_equal(x, np.zeros(3))
