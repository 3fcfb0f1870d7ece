"""Pins for the oracle's Ritz-value diagnostics (CPU, float64).

* Gauss weights against the classical product formula over the eigenvalues of
  T and of T with its first row and column removed (Golub and Meurant,
  Matrices, Moments and Quadrature, 2010): weight_i =
  prod_j (theta_i - mu_j) / prod_{k != i} (theta_i - theta_k).
* Residual bounds against the explicit residual ||A Q y_i - theta_i Q y_i||
  of a fully reorthogonalised run (A Q = Q T + beta q e_s^T).
* Ghosts: without reorthogonalisation the outlying eigenvalues of an operator
  reappear as repeated Ritz values once they converge; with full
  reorthogonalisation every eigenvalue appears once.
* The Cullum-Willoughby test flags the Ritz values of a nearly decoupled
  trailing block (zero weight, also eigenvalues of the reduced matrix) and
  no others.
"""
import numpy as np

from oracle import lanczos as OL


def test_weights_match_product_formula():
    rng = np.random.default_rng(1)
    s = 12
    a = rng.standard_normal(s)
    b = rng.uniform(0.2, 1.0, s)
    lam, w, _, _, _, _ = OL.ritz_diagnostics(a, b)
    mu = np.linalg.eigvalsh(OL.tridiag(a[1:], b[1:]))
    for i in range(s):
        num = np.prod(lam[i] - mu)
        den = np.prod(np.delete(lam[i] - lam, i))
        assert abs(w[i] - num / den) <= 1e-9 * max(w[i], 1e-12)
    assert abs(w.sum() - 1.0) <= 1e-12


def test_residual_bound_is_the_explicit_residual():
    rng = np.random.default_rng(2)
    n, m = 60, 20
    X = rng.standard_normal((n, n))
    A = (X + X.T) / 2
    a, b, Q = OL.lanczos(lambda v: A @ v, rng.standard_normal(n), m, OL.FULL)
    lam, _, resid, _, _, _ = OL.ritz_diagnostics(a, b)
    Qm = np.stack(Q[:m], 1)
    _, Y = np.linalg.eigh(OL.tridiag(a, b))
    for i in range(m):
        z = Qm @ Y[:, i]
        assert abs(np.linalg.norm(A @ z - lam[i] * z) - resid[i]) <= 1e-9 * np.abs(lam).max()


def _outlier_run(reorth):
    rng = np.random.default_rng(0)
    n = 400
    ev = np.concatenate([[100.0, 60.0, -30.0], rng.uniform(0.0, 1.0, n - 3)])
    a, b, _ = OL.lanczos(lambda v: ev * v, rng.standard_normal(n), 80, reorth)
    return OL.ritz_diagnostics(a, b, 1e-8)


def test_ghosts_without_reorthogonalisation_only():
    lam, w, resid, copies, spurious, ghosts = _outlier_run(OL.NONE)
    assert ghosts >= 2
    top = lam >= 100.0 - 1e-6
    assert copies[top].min() >= 2 and np.allclose(lam[top], 100.0, rtol=1e-10)
    # the copies share the Gauss weight of the one eigenvalue
    assert np.all(resid[top] <= 1e-8 * 100.0)
    lam, w, resid, copies, spurious, ghosts = _outlier_run(OL.FULL)
    assert ghosts == 0 and copies.max() == 1
    for x in (100.0, 60.0, -30.0):
        assert np.abs(lam - x).min() <= 1e-10 * 100.0


def test_cullum_willoughby_flags_decoupled_values():
    a = np.array([1.0, 2.0, 3.0, 4.0])
    b = np.array([0.5, 1e-15, 0.3, 0.7])
    lam, w, _, copies, spurious, ghosts = OL.ritz_diagnostics(a, b, 1e-10)
    trailing = np.linalg.eigvalsh(np.array([[3.0, 0.3], [0.3, 4.0]]))
    for x in trailing:
        i = int(np.abs(lam - x).argmin())
        assert spurious[i] and w[i] < 1e-20
    assert spurious.sum() == 2 and ghosts == 0
