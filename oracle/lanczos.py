"""Lanczos and stochastic Lanczos quadrature (oracle, float64).

Section 4 states the symmetric Lanczos recurrence
    beta_{k+1} q_{k+1} = H q_k - alpha_k q_k - beta_k q_{k-1},  alpha_k = q_k^T H q_k,
whose coefficients form the tridiagonal T_m; SLQ approximates v^T f(H) v by
e_1^T f(T_m) e_1, i.e. a Gauss quadrature with nodes the eigenvalues of T_m and
weights the squared first components of its eigenvectors.  Appendix C adds
reorthogonalisation against a sliding window of r stored vectors (one dot and
one AXPY per stored vector); section 7.1 uses full reorthogonalisation at every
iteration; section 7 (GPT-OSS run) uses none.

Readings taken where the text is loose:
* coefficient order: the standard (Paige) order of section 4 - subtract
  beta_k q_{k-1}, form alpha_k, subtract alpha_k q_k, reorthogonalise, then
  beta_{k+1} = ||w|| (Appendix C's "beta_t = ||w||" before the subtraction is
  taken as a typesetting slip);
* FULL reorthogonalisation: one modified Gram-Schmidt sweep over q_1..q_k;
  WINDOW r: the same sweep over the r most recent vectors q_{k-r+1}..q_k;
* breakdown: stop when beta_{k+1} <= tol * max_j |alpha_j| (tol 1e-12);
* outputs: alpha[0..s-1] and beta[0..s-1] = beta_2..beta_{s+1}, the last one
  being the residual norm (not part of T_s).
"""
from __future__ import annotations

import numpy as np

NONE, FULL, WINDOW = 0, 1, 2


def lanczos(hvp, q1: np.ndarray, m: int, reorth: int = FULL, window: int = 0,
            tol: float = 1e-12):
    """Run m Lanczos steps from unit vector q1.  Returns (alpha, beta, Q)."""
    q = np.asarray(q1, dtype=np.float64).copy()
    q /= np.linalg.norm(q)
    q_prev = np.zeros_like(q)
    beta_k = 0.0
    alphas, betas, basis = [], [], [q.copy()]
    for k in range(m):
        w = hvp(q) - beta_k * q_prev
        alpha = float(w @ q)
        w = w - alpha * q
        if reorth == FULL:
            sel = basis
        elif reorth == WINDOW:
            sel = basis[-window:] if window > 0 else []
        else:
            sel = []
        for qj in sel:
            w = w - float(w @ qj) * qj
        beta = float(np.linalg.norm(w))
        alphas.append(alpha)
        betas.append(beta)
        if beta <= tol * max(abs(a) for a in alphas):
            break
        q_prev, q = q, w / beta
        beta_k = beta
        basis.append(q.copy())
    return np.array(alphas), np.array(betas), basis


def tridiag(alpha, beta) -> np.ndarray:
    """Dense T_s from alpha[0..s-1] and the off-diagonals beta[0..s-2]."""
    s = len(alpha)
    T = np.diag(np.asarray(alpha, dtype=np.float64))
    for i in range(s - 1):
        T[i, i + 1] = T[i + 1, i] = beta[i]
    return T


def ritz(alpha, beta):
    """Gauss quadrature of T: nodes (Ritz values) and weights (U_1i)^2 (section 4)."""
    T = tridiag(alpha, beta)
    lam, U = np.linalg.eigh(T)
    return lam, U[0, :] ** 2


def ritz_diagnostics(alpha, beta, tol: float = 1e-8):
    """Diagnostics of the Ritz values of T_s for runs that lose orthogonality.

    Theorem 4.1 (and the GPT-OSS run of section 7, which stores no basis and
    does not reorthogonalise) concern the spurious duplicate ("ghost") Ritz
    values that appear once Lanczos vectors lose orthogonality.  Per Ritz value
    theta_i (ascending) this returns, with norm = max_i |theta_i|:
    * weight_i = (U_1i)^2, the Gauss weight;
    * resid_i = beta_{s+1} |U_si|, the residual norm ||H z_i - theta_i z_i|| of
      the Ritz pair (Paige's bound, exact while the basis is orthonormal);
    * copies_i: the size of its cluster, Ritz values chained by gaps
      <= tol * norm (a converged eigenvalue repeated by lost orthogonality);
    * spurious_i: the test of Cullum and Willoughby (Lanczos Algorithms for
      Large Symmetric Eigenvalue Computations, 1985): a simple Ritz value
      (copies_i = 1) that is also an eigenvalue of T_s with its first row and
      column removed, within tol * norm;
    and the number of ghosts, sum over clusters of (size - 1).
    """
    a = np.asarray(alpha, dtype=np.float64)
    b = np.asarray(beta, dtype=np.float64)
    s = a.size
    lam, U = np.linalg.eigh(tridiag(a, b))
    norm = float(np.abs(lam).max())
    weight = U[0, :] ** 2
    resid = abs(b[s - 1]) * np.abs(U[s - 1, :])
    copies = np.ones(s, dtype=np.int64)
    start = 0
    for i in range(1, s + 1):
        if i == s or lam[i] - lam[i - 1] > tol * norm:
            copies[start:i] = i - start
            start = i
    mu = np.linalg.eigvalsh(tridiag(a[1:], b[1:])) if s > 1 else np.zeros(0)
    spurious = np.zeros(s, dtype=bool)
    for i in range(s):
        if copies[i] == 1 and mu.size and np.abs(mu - lam[i]).min() <= tol * norm:
            spurious[i] = True
    ghosts = 0
    i = 0
    while i < s:
        ghosts += int(copies[i]) - 1
        i += int(copies[i])
    return lam, weight, resid, copies, spurious, ghosts


def slq(hvp, probes, m: int, reorth: int = FULL, window: int = 0):
    """SLQ over unit probes: per-probe nodes, weights, and tr(H) ~ P mean alpha_1."""
    nodes, weights, alpha1, steps = [], [], [], []
    P = None
    for z in probes:
        P = z.size
        a, b, _ = lanczos(hvp, z, m, reorth, window)
        lam, tau = ritz(a, b)
        nodes.append(lam)
        weights.append(tau)
        alpha1.append(a[0])
        steps.append(len(a))
    trace = P * float(np.mean(alpha1))
    return nodes, weights, trace, steps
