"""Pins for the oracle's finite-difference HVP (CPU, float64)."""
import numpy as np
import pytest

import synth
from oracle import hvp as O
from oracle import model as M
from tests import micro, torch_ref


def test_quadratic_diagonal_is_exact():
    rng = np.random.default_rng(0)
    P = 1000
    d = rng.standard_normal(P)
    theta = rng.standard_normal(P)
    v = rng.standard_normal(P)
    v /= np.linalg.norm(v)
    for eps in [1e-1, 1e-3, 1e-5]:
        hv = O.quad_diag_hvp(d, theta, v, eps)
        # Theorem 3.1: the truncation term vanishes for a quadratic (D_v^3 L = 0)
        assert np.linalg.norm(hv - d * v) <= 1e-16 / eps * 50 * np.linalg.norm(d * theta) + 1e-14


def test_quadratic_dense_is_exact():
    rng = np.random.default_rng(1)
    P = 60
    A = rng.standard_normal((P, P))
    A = A + A.T
    th = rng.standard_normal(P)
    v = rng.standard_normal(P)
    hv = O.fd_hvp(lambda t: A @ t, th, v, 1e-2)
    assert np.allclose(hv, A @ v, rtol=0, atol=1e-12 * np.abs(A @ v).max())


def test_quartic_bias_matches_theorem_3_1():
    """L = 1/4 sum c_i theta_i^4: FD - exact = eps^2/6 grad(D_v^3 L) = eps^2 c v^3 exactly."""
    rng = np.random.default_rng(2)
    P = 200
    c = rng.uniform(0.5, 2.0, P)
    th = rng.standard_normal(P)
    v = rng.standard_normal(P)
    v /= np.linalg.norm(v)
    grad = lambda t: c * t ** 3
    exact = 3 * c * th ** 2 * v
    for eps in [1e-1, 3e-2, 1e-2]:
        fd = O.fd_hvp(grad, th, v, eps)
        # D_v^3 L = sum_i 6 c_i theta_i v_i^3, whose gradient is 6 c v^3
        bias = eps ** 2 / 6 * (6 * c * v ** 3)
        # identity up to float64 rounding of the difference quotient (~1e-16 |g| / eps)
        assert np.abs(fd - exact - bias).max() <= 1e-14 / eps * np.abs(grad(th)).max() * 10
        assert np.abs(bias).max() > 1e5 * np.abs(fd - exact - bias).max()


@pytest.mark.parametrize("fam", ["gpt2", "llama"])
def test_fd_hvp_against_exact_autograd_hvp(fam):
    cfg, theta, tok = micro.inputs(micro.MICRO[fam])
    P = theta.size
    v = synth.gaussian_direction(4, P)
    exact = torch_ref.exact_hvp(micro.MICRO[fam], theta, v, tok)
    errs = []
    for eps in [1e-2, 1e-3]:
        fd = O.lm_hvp(cfg, theta, v, eps, tok)
        errs.append(np.linalg.norm(fd - exact) / np.linalg.norm(exact))
    # O(eps^2) truncation: 1e-2 -> 1e-3 shrinks the error ~100x
    assert errs[1] < 1e-5
    assert errs[0] / errs[1] > 30


@pytest.mark.parametrize("fam", ["gpt2", "llama"])
def test_hvp_symmetry(fam):
    cfg, theta, tok = micro.inputs(micro.MICRO[fam])
    P = theta.size
    v = synth.gaussian_direction(4, P)
    w = synth.gaussian_direction(5, P)
    hv = O.lm_hvp(cfg, theta, v, 1e-3, tok)
    hw = O.lm_hvp(cfg, theta, w, 1e-3, tok)
    assert abs(v @ hw - w @ hv) <= 1e-6 * np.linalg.norm(hv)


def test_dense_hessian_brute_force_micro():
    """Column-by-column Hessian from exact autograd HVPs: symmetric, and H v = FD-HVP."""
    fields = dict(micro.MICRO["gpt2"], n_layers=1, d_model=8, n_heads=2, d_ff=16, vocab=12, max_seq=6)
    cfg, theta, tok = micro.inputs(fields, batch=2, seq=6)
    P = theta.size
    assert P < 1200
    import torch
    t = torch.tensor(theta, requires_grad=True)
    (g,) = torch.autograd.grad(torch_ref.loss(fields, t, tok), t, create_graph=True)
    Hd = np.stack([torch.autograd.grad(g[j], t, retain_graph=True)[0].numpy() for j in range(P)])
    assert np.linalg.norm(Hd - Hd.T) <= 1e-10 * np.linalg.norm(Hd)
    v = synth.gaussian_direction(6, P)
    fd = O.lm_hvp(cfg, theta, v, 1e-3, tok)
    assert np.linalg.norm(fd - Hd @ v) <= 1e-5 * np.linalg.norm(Hd @ v)


def test_dataset_average_equals_concatenated_batch():
    cfg, theta, _ = micro.inputs(micro.MICRO["llama"])
    t1 = synth.tokens(10, 2, 8, cfg.vocab)
    t2 = synth.tokens(11, 3, 8, cfg.vocab)
    v = synth.gaussian_direction(7, theta.size)
    a = O.lm_hvp_dataset(cfg, theta, v, 1e-3, [t1, t2])
    b = O.lm_hvp(cfg, theta, v, 1e-3, np.concatenate([t1, t2]))
    assert np.linalg.norm(a - b) <= 1e-9 * np.linalg.norm(b)


def test_dataset_weights_are_target_counts():
    """Batches of different shapes and label masks: the weighted average of
    Algorithm 1 equals the HVP of the mean over every kept target, computed
    here on one padded batch that holds all rows (right padding with ignored
    labels does not change a row's targets, by causality)."""
    cfg, theta, _ = micro.inputs(micro.MICRO["llama"])
    t1 = synth.tokens(20, 2, 8, cfg.vocab)
    t2 = synth.tokens(21, 3, 6, cfg.vocab)
    l1 = t1.astype(np.int64).copy()
    l1[0, :3] = M.IGNORE                         # prompt mask
    l2 = t2.astype(np.int64).copy()
    l2[1, 4:] = M.IGNORE                         # padding
    v = synth.gaussian_direction(8, theta.size)
    a = O.lm_hvp_dataset(cfg, theta, v, 1e-3, [(t1, l1), (t2, l2)])
    # one batch [5, 8]: t2's rows right-padded to 8 with ignored labels
    pad = np.zeros((3, 2), dtype=t2.dtype)
    tok = np.concatenate([t1, np.concatenate([t2, pad], 1)])
    lab = np.concatenate([l1, np.concatenate([l2, np.full((3, 2), M.IGNORE)], 1)])
    b = O.lm_hvp(cfg, theta, v, 1e-3, tok, lab)
    assert M.num_targets(tok, lab) == M.num_targets(t1, l1) + M.num_targets(t2, l2)
    assert np.linalg.norm(a - b) <= 1e-8 * np.linalg.norm(b)
    # and it is not the plain average of the two batch HVPs (unequal weights)
    c = 0.5 * (O.lm_hvp(cfg, theta, v, 1e-3, t1, l1) + O.lm_hvp(cfg, theta, v, 1e-3, t2, l2))
    assert np.linalg.norm(a - c) > 1e-3 * np.linalg.norm(b)


@pytest.mark.parametrize("fam", ["gpt2", "llama"])
def test_fd_hvp_with_labels_against_exact_autograd_hvp(fam):
    cfg, theta, tok = micro.inputs(micro.MICRO[fam], seed=7)
    lab = tok.astype(np.int64).copy()
    lab[0, 6:] = M.IGNORE
    lab[1, :3] = M.IGNORE
    v = synth.gaussian_direction(9, theta.size)
    exact = torch_ref.exact_hvp(micro.MICRO[fam], theta, v, tok, lab)
    fd = O.lm_hvp(cfg, theta, v, 1e-3, tok, lab)
    assert np.linalg.norm(fd - exact) <= 1e-5 * np.linalg.norm(exact)
