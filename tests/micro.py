"""Micro model configurations and seeded inputs used by the CPU pins."""
import numpy as np

import synth
from oracle import model as M

MICRO = {
    "gpt2": dict(family="gpt2", n_layers=2, d_model=16, n_heads=2, n_kv_heads=2, d_ff=32,
                 vocab=24, max_seq=8, rope_base=10000.0),
    "llama": dict(family="llama", n_layers=2, d_model=16, n_heads=4, n_kv_heads=2, d_ff=24,
                  vocab=24, max_seq=8, rope_base=10000.0),
}


def cfg_of(fields, bf16=False):
    return M.ModelConfig(family=fields["family"], n_layers=fields["n_layers"],
                         d_model=fields["d_model"], n_heads=fields["n_heads"],
                         n_kv_heads=fields["n_kv_heads"], d_ff=fields["d_ff"],
                         vocab=fields["vocab"], max_seq=fields["max_seq"],
                         rope_base=fields["rope_base"], bf16=bf16)


def inputs(fields, batch=2, seq=8, std=0.3, seed=1, dist="uniform"):
    """Parameters with a larger init scale (so curvature is not negligible) and tokens."""
    cfg = cfg_of(fields)
    P = M.num_params(cfg)
    theta = synth.init_params(M.init_ranges(cfg), P, seed, std=std).astype(np.float64)
    # perturb gains and biases away from 1/0 so that their curvature is exercised
    for e in M.layout(cfg):
        if e.kind != M.MATRIX:
            theta[e.offset:e.offset + e.numel] += 0.1 * synth.normal(seed + 100, 1, e.offset, e.numel)
    tok = synth.tokens(seed + 1, batch, seq, fields["vocab"], dist)
    return cfg, theta, tok
