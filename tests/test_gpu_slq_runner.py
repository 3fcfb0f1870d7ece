"""The SLQ runner (`python -m paper_2602_00816_amd.slq`) end to end on the tiny
fp32 workload at its own setting (1 Rademacher probe, m = 20, full
reorthogonalisation, eps = 1e-3): its Ritz nodes, Gauss weights and trace
estimate against the oracle's Lanczos run on the same seeded inputs (section 4)."""
import json
import os

import numpy as np
import pytest

import synth.workloads
from oracle import hvp as OH
from oracle import lanczos as OL
from synth.workloads import WORKLOADS
from tests.gpu_util import need_gpu, say, workload_inputs

pytestmark = pytest.mark.gpu


def test_slq_runner_tiny_gpt2_against_oracle(tmp_path):
    need_gpu()
    from paper_2602_00816_amd import slq
    w = WORKLOADS["tiny-gpt2-fp32"]
    out_file = os.path.join(tmp_path, "slq.json")
    got = slq.main(["--workload", "tiny-gpt2-fp32", "--out", out_file])
    assert json.load(open(out_file))["lanczos_steps"] == got["lanczos_steps"]
    cfg, theta, tok = workload_inputs(w)
    P = theta.size
    m, eps = w["m"], w["eps"][0]
    assert got["params"] == P and got["probes"] == 1 and got["m"] == m
    q1 = synth.rademacher_probe(synth.workloads.SEED_PROBE, P).astype(np.float64)
    ao, bo, _ = OL.lanczos(lambda x: OH.lm_hvp(cfg, theta, x, eps, tok), q1, m, OL.FULL)
    lo, to = OL.ritz(ao, bo)
    nodes, weights = np.array(got["nodes"][0]), np.array(got["weights"][0])
    assert nodes.size == m
    scale = np.abs(lo).max()
    say(f"runner Ritz [{nodes.min():.6e}, {nodes.max():.6e}] vs oracle [{lo.min():.6e}, {lo.max():.6e}]; "
        f"trace {got['trace_estimate']:.6e} vs {P * ao[0]:.6e}")
    assert abs(nodes.max() - lo.max()) <= 1e-3 * scale
    assert abs(nodes.min() - lo.min()) <= 1e-3 * scale
    assert abs(weights.sum() - 1.0) < 1e-9
    # the weight of the largest Ritz value: the squared first component of its eigenvector
    assert abs(weights[np.argmax(nodes)] - to[np.argmax(lo)]) <= 1e-3
    assert abs(got["trace_estimate"] - P * ao[0]) <= 1e-4 * abs(P * ao[0]) + 1e-6 * scale * P
    assert abs(sum(got["density_mass"]) - 1.0) < 1e-9
