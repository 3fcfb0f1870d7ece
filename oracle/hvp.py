"""Central finite-difference Hessian-vector product (oracle, float64).

Section 3.1, Eq. (grad-fd-hvp): Hv is approximated by the difference of the
gradients at theta + eps v and theta - eps v, divided by 2 eps.  Algorithm 1
accumulates, over the batches of a dataloader, w_b times the gradient of the
batch loss at the + point and minus the same at the - point, then divides by
2 eps sum_b w_b.  The reading used here: w_b is the number of target tokens of
batch b (a token-weighted mean), and the division is by 2 eps sum_b w_b (the
algorithm's last step is garbled; the text after it states the (2 eps)^-1
scaling).  theta itself is never modified: the two points are formed out of
place, so no restore step is needed.
"""
from __future__ import annotations

import numpy as np

from . import model as M


def fd_hvp(grad_fn, theta: np.ndarray, v: np.ndarray, eps: float) -> np.ndarray:
    """(grad(theta + eps v) - grad(theta - eps v)) / (2 eps), all float64."""
    theta = np.asarray(theta, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    gp = grad_fn(theta + eps * v)
    gm = grad_fn(theta - eps * v)
    return (gp - gm) / (2.0 * eps)


def lm_grad_fn(cfg: M.ModelConfig, tokens: np.ndarray, labels=None):
    def g(th):
        return M.loss_and_grad(cfg, th, tokens, labels=labels)[1]
    return g


def lm_hvp(cfg: M.ModelConfig, theta, v, eps: float, tokens, labels=None) -> np.ndarray:
    """FD-HVP of the mean next-token loss on one batch (Algorithm 1, one batch)."""
    return fd_hvp(lm_grad_fn(cfg, tokens, labels), theta, v, eps)


def lm_hvp_dataset(cfg: M.ModelConfig, theta, v, eps: float, batches) -> np.ndarray:
    """Algorithm 1 over several batches with token weights w_b = the number of
    targets of batch b.

    ``batches`` holds token arrays [B_b, S_b] or (tokens, labels) pairs (labels
    as in model.loss_and_grad).  Each batch loss is a mean over its own targets,
    so w_b times its gradient is the gradient of the summed loss; dividing by
    2 eps sum_b w_b gives the HVP of the token-weighted mean loss over all
    batches.
    """
    theta = np.asarray(theta, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    items = [b if isinstance(b, tuple) else (b, None) for b in batches]
    acc = np.zeros_like(theta)
    wsum = 0.0
    tp = theta + eps * v
    for tok, lab in items:
        w = M.num_targets(tok, lab)
        acc += w * M.loss_and_grad(cfg, tp, tok, labels=lab)[1]
        wsum += w
    tm = theta - eps * v
    for tok, lab in items:
        w = M.num_targets(tok, lab)
        acc -= w * M.loss_and_grad(cfg, tm, tok, labels=lab)[1]
    return acc / (2.0 * eps * wsum)


# ----------------------------------------------------------------------------
# quadratic-diagonal operator: L(theta) = 1/2 sum_i d_i theta_i^2
# ----------------------------------------------------------------------------
def quad_diag_grad_fn(diag: np.ndarray):
    dd = np.asarray(diag, dtype=np.float64)

    def g(th):
        return dd * th
    return g


def quad_diag_hvp(diag, theta, v, eps: float) -> np.ndarray:
    """FD-HVP of the diagonal quadratic; equals diag * v in exact arithmetic."""
    return fd_hvp(quad_diag_grad_fn(diag), theta, v, eps)
