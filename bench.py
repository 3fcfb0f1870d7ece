"""Benchmark of the FD-HVP + Lanczos hot path on one MI355X.

A step is one Lanczos iteration (section 4) of the Llama-style 1.3B bf16
workload: one finite-difference HVP (two gradient passes in lockstep over a
4 x 2048 Zipf(1.1) token batch, eps = 1e-3), the three-term recurrence and
full classical Gram-Schmidt (twice) reorthogonalisation against the bf16
Krylov basis.  The timed region is one fdh_lanczos call of K steps, so the
reorthogonalisation cost is averaged over k = 1..K as in a real run; it runs
without per-launch instrumentation.  A second, instrumented run of the same K
steps (HIP events around every launch on the context stream) gives the
per-family breakdown and the GEMM roofline.  One full SLQ probe at the
workload's own Lanczos length (m = 40 for the 1.3B workload) is timed after
that, whatever K is.

Prints one JSON line.  `value` is FD-HVPs per second through the timed
Lanczos steps (each step performs exactly one HVP); Lanczos iterations per
minute, HVP-only throughput, the SLQ probe, the GEMM roofline and the oracle's
CPU rate are reported beside it.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from synth.workloads import WORKLOADS, SEED_PARAMS, SEED_TOKENS, SEED_PROBE  # noqa: E402

METRIC = "FD-HVPs/sec + Lanczos iters/min at 1.3B bf16; MFMA util % / HBM GB/s"
PEAK_BF16_TFLOPS = 2500.0
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBPS = 8000.0


def alg_flops_per_hvp(w: dict) -> tuple[float, float]:
    """Algorithmic FLOPs of one HVP, split into (weight products, attention
    products): two gradient passes of 6 N_mm T and 3 A_fwd each."""
    d, F, V, L = w["d_model"], w["d_ff"], w["vocab"], w["n_layers"]
    H, Hk = w["n_heads"], w["n_kv_heads"]
    dh = d // H
    B, S = w["batch"], w["seq"]
    T = B * S
    if w["family"] == "llama":
        per_layer = d * (H + 2 * Hk) * dh + H * dh * d + d * 2 * F + F * d
    else:
        per_layer = d * 3 * d + d * d + d * F + F * d
    n_mm = L * per_layer + d * V
    a_fwd = L * 2.0 * B * H * S * S * dh      # causal QK^T and PV
    return 2.0 * 6.0 * n_mm * T, 2.0 * 3.0 * a_fwd


def committed_gemm_traffic(workload: str):
    """HBM bytes per step of the GEMM launches, from the committed counter
    summary, or None when the GEMM source changed after the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"gemm_{workload}.md")
    src = os.path.join(ROOT, "paper_2602_00816_amd", "csrc", "gemm.hip")
    try:
        txt = open(path).read()
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    except OSError:
        return None
    vals = dict(l.split(": ", 1) for l in txt.splitlines() if l.startswith(("traffic_bytes_per_step:", "gemm_source_sha256:")))
    if vals.get("gemm_source_sha256", "").strip() != sha:
        return None
    return float(vals["traffic_bytes_per_step"])


def cpu_baseline(w: dict, budget_s: float = 20.0) -> dict:
    """The fp64 oracle's HVP on a bounded slice of the workload, scaled by FLOPs."""
    from oracle import hvp as OH
    from oracle import model as M
    import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([t.get("num_threads", 1) for t in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    sample = dict(w, n_layers=2, batch=1, seq=1024)
    cfg = M.ModelConfig(family=sample["family"], n_layers=2, d_model=w["d_model"], n_heads=w["n_heads"],
                        n_kv_heads=w["n_kv_heads"], d_ff=w["d_ff"], vocab=w["vocab"], max_seq=w["max_seq"],
                        rope_base=w["rope_base"], bf16=True)
    P = M.num_params(cfg)
    theta = synth.init_params(M.init_ranges(cfg), P, SEED_PARAMS, bf16=True).astype(np.float64)
    tok = synth.tokens(SEED_TOKENS, 1, 1024, w["vocab"], w["token_dist"])
    v = synth.rademacher_probe(SEED_PROBE, P).astype(np.float64)
    t0 = time.perf_counter()
    OH.lm_hvp(cfg, theta, v, 1e-3, tok)
    dt = time.perf_counter() - t0
    scale = sum(alg_flops_per_hvp(w)) / sum(alg_flops_per_hvp(sample))
    return {"value": 1.0 / (dt * scale), "unit": "FD-HVPs/s", "cores": int(threads), "kind": "oracle, extrapolated",
            "sample": f"{w['family']} d={w['d_model']} with 2 of {w['n_layers']} layers, 1x1024 tokens, "
                      f"fp64 numpy HVP {dt:.2f} s, scaled x{scale:.1f} by algorithmic FLOPs to the full workload"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40, help="timed Lanczos steps")
    ap.add_argument("--warmup", type=int, default=2, help="untimed HVPs before the timed run")
    ap.add_argument("--workload", default="llama-1.3b-bf16")
    ap.add_argument("--hvp-reps", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cg-steps", type=int, default=2, help="timed CG inverse-HVP steps after the Lanczos run")
    ap.add_argument("--slq-m", type=int, default=-1,
                    help="Lanczos length of the timed SLQ probe (-1: the workload's m, 0: no probe)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run one plain 1 GiB device copy first (reference for hardware byte counters)")
    args = ap.parse_args()
    args.hvp_reps = max(1, args.hvp_reps)
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on exactly one GPU: this build has no multi-GPU path "
              "(the sharded design is described, not built).", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2602_00816_amd import fdhvp as fd

    w = WORKLOADS[args.workload]
    K, W = args.steps, args.warmup
    eps = w["eps"][0]
    B, S = w["batch"], w["seq"]
    mod = fd.Model.from_workload(w)
    o = fd.opts(w["reorth"], w["window"], w["basis"])
    m_slq = int(w["m"]) if args.slq_m < 0 else args.slq_m
    m_plan = max(K, 2, m_slq)
    ws = mod.set_workspace(B, S, m_plan, o)
    params = mod.init_params(SEED_PARAMS)
    tok = mod.make_tokens(B, S, SEED_TOKENS, w["token_dist"])
    v = mod.random_vector(SEED_PROBE, "rademacher")
    hv = torch.empty_like(v)
    mod.bind(params, tok, eps)
    torch.cuda.synchronize()
    print(f"[bench] {args.workload}: P={mod.num_params} workspace={ws / 1e9:.1f} GB", file=sys.stderr, flush=True)
    if args.copy_calibration:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        fd.testing_copy(dst, src, 1 << 30)
        torch.cuda.synchronize()
        del src, dst
        print("[bench] copy calibration: 1 GiB copied", file=sys.stderr, flush=True)

    for i in range(W):
        mod.hvp(params, v, eps, tok, out=hv)
    mod.lanczos(2, SEED_PROBE, o)
    torch.cuda.synchronize()
    print("[bench] warmup done", file=sys.stderr, flush=True)

    # HVP-only throughput
    t0 = time.perf_counter()
    for i in range(args.hvp_reps):
        mod.hvp(params, v, eps, tok, out=hv)
    torch.cuda.synchronize()
    t_hvp = (time.perf_counter() - t0) / args.hvp_reps
    print(f"[bench] hvp {t_hvp * 1e3:.1f} ms", file=sys.stderr, flush=True)

    # the timed Lanczos steps (no instrumentation)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    alpha, beta, steps, st = mod.lanczos(K, SEED_PROBE, o)
    torch.cuda.synchronize()
    t_total = time.perf_counter() - t0
    print(f"[bench] lanczos {K} steps {t_total:.2f} s (steps_done {steps})", file=sys.stderr, flush=True)

    # the same K steps again, with HIP events around every launch on the context stream
    mod.timing(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    mod.lanczos(K, SEED_PROBE, o)
    torch.cuda.synchronize()
    t_instr = time.perf_counter() - t0
    tm = mod.timing_read()
    mod.timing(False)
    print(f"[bench] instrumented run {K} steps {t_instr:.2f} s", file=sys.stderr, flush=True)

    # one full SLQ probe at the workload's Lanczos length
    slq = None
    if m_slq > 0:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        nodes, weights, slq_steps, trace, _ = mod.slq_density(1, m_slq, SEED_PROBE, o)
        torch.cuda.synchronize()
        t_slq = time.perf_counter() - t0
        print(f"[bench] slq probe m={m_slq} {t_slq:.2f} s", file=sys.stderr, flush=True)
        n = int(slq_steps[0])
        slq = {"m": m_slq, "steps_done": n, "seconds": t_slq, "lanczos_iters_per_min": 60.0 * n / t_slq,
               "hvp_per_s": n / t_slq, "ritz_max": float(nodes[0, :n].max()), "ritz_min": float(nodes[0, :n].min()),
               "trace_estimate": trace}

    ms_step = t_total * 1e3 / K
    value = K / t_total
    alg_mm, alg_att = alg_flops_per_hvp(w)
    alg = alg_mm + alg_att
    gemm_ms_per_step = tm["gemm"]["ms"] / K
    fused = bool(tm["attention"]["launches"] > 0)
    # with fused attention the GEMMs carry only the weight products
    alg_gemm = alg_mm if fused else alg
    achieved = alg_gemm / (gemm_ms_per_step * 1e-3) / 1e12
    att_ms_per_step = tm["attention"]["ms"] / K
    executed = tm["gemm"]["flops"] / (tm["gemm"]["ms"] * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if w["dtype"] == "bf16" else PEAK_F32_TFLOPS
    lz_gbps = tm["lanczos"]["bytes"] / (tm["lanczos"]["ms"] * 1e-3) / 1e9 if tm["lanczos"]["ms"] > 0 else None
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "FD-HVPs/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w["dtype"],
        "data": "synthetic (N(0,0.02) weights, Zipf(1.1) tokens, seeded)",
        "config": {"workload": args.workload, "params": mod.num_params, "global_batch": B, "seq_len": S,
                   "eps": eps, "lanczos_m": K, "reorth": w["reorth"], "basis": w["basis"], "parallelism": "none"},
        "lanczos_iters_per_min": 60.0 * value,
        "ms_per_step_instrumented": t_instr * 1e3 / K,
        "slq_probe": slq,
        "hvp_only_per_s": 1.0 / t_hvp,
        "hvp_tokens_per_s": B * S / t_hvp,
        "lanczos_overhead": (ms_step * 1e-3) / t_hvp - 1.0,
        "gemm_ms_per_step": gemm_ms_per_step,
        "gemm_launches_per_step": tm["gemm"]["launches"] / K,
        "mfma_util_executed": executed / peak,
        "model_flop_util": alg / (ms_step * 1e-3) / 1e12 / peak,
        "attention_fused": fused,
        "attention_ms_per_step": att_ms_per_step if fused else None,
        "attention_tflops": (alg_att / (att_ms_per_step * 1e-3) / 1e12) if fused else None,
        "lanczos_vec_ms_per_step": tm["lanczos"]["ms"] / K,
        "lanczos_vec_hbm_GBps": lz_gbps,
        "lanczos_vec_hbm_frac": (lz_gbps / PEAK_HBM_GBPS) if lz_gbps else None,
        "roofline": {"bound": "mfma", "kernel": "bf16 MFMA GEMM (all launches of one step, instrumented run)",
                     "achieved": achieved, "peak": peak, "unit": "TFLOP/s", "frac": achieved / peak,
                     "traffic": committed_gemm_traffic(args.workload)},
    }
    if args.cg_steps > 0:
        # damped CG (H + lam I) x = b, lam well above the extreme Ritz values of the run
        # (three times the largest Ritz value magnitude of the timed run)
        from scipy.linalg import eigh_tridiagonal
        ritz = eigh_tridiagonal(alpha[:steps], beta[:max(steps - 1, 0)], eigvals_only=True)
        lam = 3.0 * float(np.abs(ritz).max())
        b = mod.random_vector(SEED_PROBE + 1, "gaussian")
        mod.timing(True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        _, res, cs, cst = mod.cg_solve(b, lam, args.cg_steps, 0.0)
        torch.cuda.synchronize()
        t_cg = time.perf_counter() - t0
        tc = mod.timing_read()
        mod.timing(False)
        print(f"[bench] cg {cs} steps {t_cg:.2f} s", file=sys.stderr, flush=True)
        vms = tc["lanczos"]["ms"]
        out["cg"] = {"steps": cs, "status": cst, "lambda": lam, "ms_per_step": t_cg * 1e3 / max(cs, 1),
                     "vec_ms_per_step": vms / max(cs, 1),
                     "vec_hbm_GBps": tc["lanczos"]["bytes"] / (vms * 1e-3) / 1e9 if vms > 0 else None,
                     "residual_ratio": float(res[-1] / res[0])}
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
