"""Helpers shared by the GPU tests: device checks, uploads, oracle-side inputs."""
import sys

import numpy as np
import pytest

import synth
from oracle import model as M
from tests import micro


def need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2602_00816_amd import fdhvp
    fdhvp.lib()  # fails loudly when the HIP library is missing
    return torch


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def upload_params(torch, theta_f32: np.ndarray, dtype: str):
    t = torch.from_numpy(np.ascontiguousarray(theta_f32, dtype=np.float32)).cuda()
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def workload_inputs(w: dict, batch=None, seq=None, std=0.02, seed_params=1, seed_tokens=2):
    """Oracle config, float32 theta (bf16-exact for bf16 workloads) and tokens."""
    cfg = micro.cfg_of(w, bf16=w["dtype"] == "bf16")
    P = M.num_params(cfg)
    theta = synth.init_params(M.init_ranges(cfg), P, seed_params, std=std, bf16=w["dtype"] == "bf16")
    tok = synth.tokens(seed_tokens, batch or w["batch"], seq or w["seq"], w["vocab"], w["token_dist"])
    return cfg, theta, tok


def rel_l2(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))
