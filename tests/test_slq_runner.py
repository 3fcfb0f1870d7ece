"""Host logic of the SLQ runner (no GPU): the binned density keeps the mass of
the Gauss weights and its bins span the Ritz values."""
import numpy as np

from paper_2602_00816_amd.slq import density_bins


def test_density_bins_conserve_mass_and_span_nodes():
    rng = np.random.default_rng(0)
    probes, m = 3, 12
    nodes = np.sort(rng.normal(size=(probes, m)) * 10, axis=1)
    w = rng.random((probes, m))
    w /= w.sum(axis=1, keepdims=True)
    steps = np.array([12, 9, 12])
    for p in range(probes):
        w[p, steps[p]:] = 0.0
        w[p] /= w[p].sum()
    edges, mass = density_bins(nodes, w, steps, nbins=7)
    assert np.isclose(mass.sum(), 1.0, atol=1e-12)
    used = np.concatenate([nodes[p, :steps[p]] for p in range(probes)])
    assert edges[0] == used.min() and edges[-1] == used.max()
    # a single node: one bin holds all the mass
    e1, m1 = density_bins(np.array([[2.0]]), np.array([[1.0]]), np.array([1]), nbins=4)
    assert np.isclose(m1.sum(), 1.0) and e1[0] == 2.0
