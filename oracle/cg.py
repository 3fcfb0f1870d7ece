"""Conjugate-gradient inverse-HVP solver (oracle, float64).

Test infrastructure only: the product path never imports this module.

The paper names CG-based inverse-HVP solvers as a consumer of the HVP
primitive with the same cost structure as Lanczos (introduction, list of
contributions; section 4, cost model): repeated HVP calls, scalar reductions
and vector updates.  It gives no algorithm of its own, so this is the method
of Hestenes and Stiefel (J. Res. NBS 49, 1952) for the damped system
    (H + lam I) x = b,   x_0 = 0,
in its textbook form:
    r_0 = b, p_0 = r_0
    alpha_k = (r_k, r_k) / (p_k, A p_k)
    x_{k+1} = x_k + alpha_k p_k,   r_{k+1} = r_k - alpha_k A p_k
    beta_k = (r_{k+1}, r_{k+1}) / (r_k, r_k),   p_{k+1} = r_{k+1} + beta_k p_k
Readings taken where the text is silent:
* stopping: after max_iters steps, or as soon as ||r_{k+1}|| <= rel_tol ||b||;
* breakdown: (p, A p) <= 0 (A not positive definite along p; possible for an
  indefinite Hessian with too small a damping) stops before the update, with
  x_k returned;
* outputs: x, the number of completed steps and the residual norms
  ||r_0||, ||r_1||, ... of the completed steps.
"""
from __future__ import annotations

import numpy as np

OK, BREAKDOWN = 0, 1


def cg(hvp, b: np.ndarray, lam: float, max_iters: int, rel_tol: float = 0.0):
    """Solve (H + lam I) x = b by CG from x_0 = 0.

    hvp: callable v -> H v (float64).  Returns (x, steps, res_norms, status)."""
    b = np.asarray(b, dtype=np.float64)
    x = np.zeros_like(b)
    r = b.copy()
    p = r.copy()
    rr = float(r @ r)
    bnorm = np.sqrt(rr)
    res = [bnorm]
    status = OK
    steps = 0
    for _ in range(max_iters):
        ap = hvp(p) + lam * p
        pap = float(p @ ap)
        if not pap > 0.0:
            status = BREAKDOWN
            break
        alpha = rr / pap
        x = x + alpha * p
        r = r - alpha * ap
        rr_new = float(r @ r)
        steps += 1
        res.append(np.sqrt(rr_new))
        if np.sqrt(rr_new) <= rel_tol * bnorm:
            break
        p = r + (rr_new / rr) * p
        rr = rr_new
    return x, steps, np.array(res), status
