"""Writes the fp64 oracle's expected values for the parity tests at the bf16
workloads' real token batches (full width and vocabulary, reduced depth) and
for the small fp32 workload's full Lanczos run.

Only the oracle (``oracle/``) and the seeded input generator (``synth``) are
called; nothing here comes from the HIP library.  At these sizes one oracle
FD-HVP takes minutes and its output is a vector of up to 1.5e9 entries, so
each case keeps a compact record of every product the parity test compares:

* per parameter block (the layout entries): the exact squared norm of the
  block of Hv, the values of Hv at up to ``NSAMPLE`` sampled indices of the
  block (drawn once, stored with the values), and the block's inner products
  with ``NSKETCH`` seeded Rademacher vectors (every entry of the block takes
  part in those, so a sketch of the block's error is available without the
  full vector);
* for the Lanczos probe: the oracle's first Lanczos coefficients alpha_1 and
  beta_2 (section 4), which fix the second Krylov vector.

Directions: ``probe`` = the Rademacher probe z/sqrt(P) of seed 3 (the SLQ
probe q_1), ``gauss`` = the Gaussian unit direction of seed 4.

Usage: python tests/golden/make_scale_fixtures.py [--out DIR] CASE [CASE ...]
       python tests/golden/make_scale_fixtures.py --list
Each case is written to DIR/<case>.npz (default tests/golden/scale).  The 8B
case needs about 90 GB of host memory.
"""
from __future__ import annotations

import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import synth  # noqa: E402
from oracle import hvp as OH  # noqa: E402
from oracle import lanczos as OL  # noqa: E402
from oracle import model as M  # noqa: E402
from synth.workloads import SEED_GAUSS, SEED_PARAMS, SEED_PROBE, SEED_TOKENS, WORKLOADS  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "scale")
NSAMPLE = 2048
NSKETCH = 16
SKETCH_SEED0 = 1000   # Rademacher sign vectors of seeds 1000 .. 1015 (probe stream)
EPS = 1e-3

# name -> workload, overrides, token batch, directions, Lanczos coefficients
CASES = {
    "llama-1.3b-2l-4x2048": dict(workload="llama-1.3b-bf16", n_layers=2, batch=4, seq=2048,
                                 dirs=("probe", "gauss"), lanczos=True),
    "gpt2-medium-2l-8x1024": dict(workload="gpt2-medium-bf16", n_layers=2, batch=8, seq=1024,
                                  dirs=("probe", "gauss"), lanczos=True),
    "llama3-8b-2l-1x2048": dict(workload="llama3-8b-bf16", n_layers=2, batch=1, seq=2048,
                                dirs=("probe",), lanczos=True),
}
for _L in (1, 2, 4, 8, 16, 24):
    CASES[f"llama-1.3b-depth{_L}-1x2048"] = dict(workload="llama-1.3b-bf16", n_layers=_L, batch=1, seq=2048,
                                                 dirs=("probe",), lanczos=False)
# the small fp32 workload's SLQ setting, one probe: m = 80 steps, full reorthogonalisation
LANCZOS_CASES = {
    "small-gpt2-lanczos-m80": dict(workload="small-gpt2-fp32", m=80),
}


def model_cfg(w: dict) -> M.ModelConfig:
    return M.ModelConfig(family=w["family"], n_layers=w["n_layers"], d_model=w["d_model"], n_heads=w["n_heads"],
                         n_kv_heads=w["n_kv_heads"], d_ff=w["d_ff"], vocab=w["vocab"], max_seq=w["max_seq"],
                         rope_base=w["rope_base"], bf16=w["dtype"] == "bf16")


def inputs(w: dict, batch: int, seq: int):
    cfg = model_cfg(w)
    P = M.num_params(cfg)
    theta = synth.init_params(M.init_ranges(cfg), P, SEED_PARAMS, bf16=w["dtype"] == "bf16")
    tok = synth.tokens(SEED_TOKENS, batch, seq, w["vocab"], w["token_dist"])
    return cfg, theta, tok


def direction(kind: str, P: int) -> np.ndarray:
    if kind == "probe":
        return synth.rademacher_probe(SEED_PROBE, P).astype(np.float64)
    return synth.gaussian_direction(SEED_GAUSS, P)


def log(*a):
    print(*a, flush=True)


def oracle_hvp(cfg, theta, v, tok, tag):
    """oracle.hvp.lm_hvp, with a line printed after each of its two gradients
    (one gradient of the larger cases takes minutes)."""
    g = OH.lm_grad_fn(cfg, tok)
    n = [0]

    def grad(th):
        t = time.time()
        r = g(th)
        n[0] += 1
        log(f"  {tag}: gradient {n[0]} of 2 ({time.time() - t:.1f} s)")
        return r
    return OH.fd_hvp(grad, theta, v, EPS)


def hvp_case(name: str, spec: dict):
    w = dict(WORKLOADS[spec["workload"]], n_layers=spec["n_layers"])
    t0 = time.time()
    cfg, theta, tok = inputs(w, spec["batch"], spec["seq"])
    P = theta.size
    lay = M.layout(cfg)
    log(f"[{name}] P={P} inputs {time.time() - t0:.1f} s")
    rng = np.random.default_rng(20260)
    rec = dict(P=np.int64(P), eps=np.float64(EPS), batch=np.int64(spec["batch"]), seq=np.int64(spec["seq"]),
               n_layers=np.int64(spec["n_layers"]), workload=np.array(spec["workload"]),
               entry_names=np.array([e.name for e in lay]), entry_offsets=np.array([e.offset for e in lay], np.int64),
               entry_numels=np.array([e.numel for e in lay], np.int64), dirs=np.array(spec["dirs"]),
               nsketch=np.int64(NSKETCH), sketch_seed0=np.int64(SKETCH_SEED0))
    for i, e in enumerate(lay):
        k = min(e.numel, NSAMPLE)
        rec[f"idx{i}"] = np.sort(rng.choice(e.numel, size=k, replace=False)).astype(np.uint32)
    for kind in spec["dirs"]:
        v = direction(kind, P)
        t1 = time.time()
        if kind == "probe" and spec["lanczos"]:
            cache = {}

            def hv_fn(x):
                cache["hv"] = oracle_hvp(cfg, theta, x, tok, f"{name} {kind}")
                return cache["hv"]
            a, b, _ = OL.lanczos(hv_fn, v, 1, OL.FULL)
            hv = cache["hv"]
            rec["alpha1"] = np.float64(a[0])
            rec["beta2"] = np.float64(b[0])
        else:
            hv = oracle_hvp(cfg, theta, v, tok, f"{name} {kind}")
        log(f"[{name}] {kind}: oracle FD-HVP {time.time() - t1:.1f} s, ||Hv|| = {np.linalg.norm(hv):.6e}")
        del v
        rec[f"{kind}_norm2"] = np.array([float(hv[e.offset:e.offset + e.numel] @ hv[e.offset:e.offset + e.numel])
                                         for e in lay])
        for i, e in enumerate(lay):
            rec[f"{kind}_val{i}"] = hv[e.offset + rec[f"idx{i}"].astype(np.int64)]
        sk = np.zeros((NSKETCH, len(lay)))
        for j in range(NSKETCH):
            if j % 4 == 0:
                log(f"  {name} {kind}: sketch {j} of {NSKETCH}")
            z = synth.rademacher(SKETCH_SEED0 + j, P)
            for i, e in enumerate(lay):
                sk[j, i] = float(hv[e.offset:e.offset + e.numel] @ z[e.offset:e.offset + e.numel])
            del z
        rec[f"{kind}_sketch"] = sk
        del hv
    os.makedirs(OUT, exist_ok=True)
    np.savez_compressed(os.path.join(OUT, name + ".npz"), **rec)
    log(f"[{name}] written ({time.time() - t0:.1f} s)")


def lanczos_case(name: str, spec: dict):
    w = WORKLOADS[spec["workload"]]
    t0 = time.time()
    cfg, theta, tok = inputs(w, w["batch"], w["seq"])
    P = theta.size
    q1 = synth.rademacher_probe(SEED_PROBE, P).astype(np.float64)
    n = [0]

    def hv_fn(x):
        n[0] += 1
        t = time.time()
        r = OH.lm_hvp(cfg, theta, x, EPS, tok)
        log(f"[{name}] step {n[0]}: {time.time() - t:.1f} s")
        return r
    a, b, _ = OL.lanczos(hv_fn, q1, spec["m"], OL.FULL)
    os.makedirs(OUT, exist_ok=True)
    np.savez_compressed(os.path.join(OUT, name + ".npz"), P=np.int64(P), eps=np.float64(EPS), m=np.int64(spec["m"]),
                        workload=np.array(spec["workload"]), alpha=a, beta=b)
    log(f"[{name}] written, {len(a)} steps ({time.time() - t0:.1f} s)")


def main(argv):
    global OUT
    if len(argv) >= 2 and argv[0] == "--out":
        OUT = os.path.abspath(argv[1])
        argv = argv[2:]
    if not argv or argv[0] == "--list":
        for k in list(CASES) + list(LANCZOS_CASES):
            print(k)
        return 0
    for name in argv:
        if name in CASES:
            hvp_case(name, CASES[name])
        elif name in LANCZOS_CASES:
            lanczos_case(name, LANCZOS_CASES[name])
        else:
            raise SystemExit(f"unknown case {name}")
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
