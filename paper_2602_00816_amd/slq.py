"""Stochastic Lanczos quadrature of a workload's loss Hessian on one GPU.

    python -m paper_2602_00816_amd.slq --workload llama-1.3b-bf16 [--probes N] [--m M]
                                       [--eps E] [--block-diagonal] [--out FILE.json]

Runs the SLQ estimate of section 4 with the workload's own settings (probe
count, Lanczos length, reorthogonalisation mode and window, basis precision,
finite-difference step, activation recomputation) on its synthetic inputs: random-init weights and a
Zipf(1.1) token batch from the workload seeds.  Every probe is a Rademacher
vector; each Lanczos step is one FD-HVP (section 3.1) through the library.

Prints, per probe, the steps completed and the extreme Ritz values, then the
trace estimate P * mean(alpha_1) and the spectral density as Gauss weights
summed into bins (the density of section 4 is the average over probes of
sum_j tau_j delta(lambda - theta_j)).  Where the workload reorthogonalises
against a window (or not at all) it repeats probe 0 for its (alpha, beta)
and flags the ghost copies among the Ritz values.  With --block-diagonal it
also forms, for a Gaussian unit direction v, the layer-block-diagonal product
(v restricted to each layer's block, the proxy of section 6, Exp I) and
reports its relative error and cosine against the full Hv per layer.  --out
writes everything as JSON.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from synth.workloads import WORKLOADS, SEED_PARAMS, SEED_TOKENS, SEED_PROBE, SEED_GAUSS  # noqa: E402


def density_bins(nodes, weights, steps, nbins=40):
    """Average over probes of the Gauss weights summed into nbins equal bins
    spanning the Ritz values of all probes: (edges, mass)."""
    th = np.concatenate([nodes[p, :steps[p]] for p in range(len(steps))])
    tw = np.concatenate([weights[p, :steps[p]] for p in range(len(steps))]) / len(steps)
    lo, hi = float(th.min()), float(th.max())
    if hi <= lo:
        hi = lo + 1.0
    edges = np.linspace(lo, hi, nbins + 1)
    mass, _ = np.histogram(th, bins=edges, weights=tw)
    return edges, mass


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", default="llama-1.3b-bf16", choices=sorted(WORKLOADS))
    ap.add_argument("--probes", type=int, default=-1, help="Rademacher probes (-1: the workload's)")
    ap.add_argument("--m", type=int, default=-1, help="Lanczos steps per probe (-1: the workload's)")
    ap.add_argument("--eps", type=float, default=-1.0, help="finite-difference step (-1: the workload's first)")
    ap.add_argument("--seed", type=int, default=SEED_PROBE, help="probe seed")
    ap.add_argument("--block-diagonal", action="store_true", help="also the layer-block-diagonal proxy (Exp I)")
    ap.add_argument("--out", default="", help="write the results as JSON")
    args = ap.parse_args(argv)

    import torch
    from paper_2602_00816_amd import fdhvp as fd

    w = WORKLOADS[args.workload]
    probes = w["probes"] if args.probes < 0 else args.probes
    m = w["m"] if args.m < 0 else args.m
    eps = w["eps"][0] if args.eps < 0 else args.eps
    B, S = w["batch"], w["seq"]
    o = fd.opts(w["reorth"], w["window"], w["basis"])
    say = lambda s: print(f"[slq] {s}", flush=True)

    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    mod = fd.Model.from_workload(w)
    mod.set_recompute(w.get("recompute", False))
    ws = mod.set_workspace(B, S, m, o)
    params = mod.init_params(SEED_PARAMS)
    tok = mod.make_tokens(B, S, SEED_TOKENS, w["token_dist"])
    mod.bind(params, tok, eps)
    torch.cuda.synchronize()
    say(f"{args.workload}: P = {mod.num_params}, {B}x{S} tokens, eps {eps:g}, {probes} probes x m = {m}, "
        f"reorth {w['reorth']}{' ' + str(w['window']) if w['reorth'] == 'window' else ''}, {w['basis']} basis, "
        f"workspace {ws / 1e9:.1f} GB{' (activation recomputation)' if w.get('recompute') else ''}")

    t0 = time.perf_counter()
    nodes, weights, steps, trace, st = mod.slq_density(probes, m, args.seed, o)
    torch.cuda.synchronize()
    t = time.perf_counter() - t0
    n_hvp = int(steps.sum())
    say(f"SLQ done in {t:.1f} s: {n_hvp} Lanczos steps, {60.0 * n_hvp / t:.1f} iters/min, status {st}")
    per_probe = []
    for p in range(probes):
        s = int(steps[p])
        th = nodes[p, :s]
        per_probe.append(dict(steps=s, ritz_min=float(th.min()), ritz_max=float(th.max()),
                              weight_sum=float(weights[p, :s].sum())))
        say(f"probe {p}: {s} steps, Ritz [{th.min():.6e}, {th.max():.6e}], sum of weights {weights[p, :s].sum():.12f}")
    edges, mass = density_bins(nodes, weights, steps)
    say(f"trace estimate {trace:.6e}")
    say("density (bin centre, mass): " + ", ".join(f"({0.5 * (edges[i] + edges[i + 1]):.3e}, {mass[i]:.3e})"
                                                   for i in range(len(mass)) if mass[i] > 0))
    out = dict(workload=args.workload, params=mod.num_params, batch=B, seq=S, eps=eps, probes=probes, m=m,
               reorth=w["reorth"], window=w["window"], basis=w["basis"], seconds=t, lanczos_steps=n_hvp,
               iters_per_min=60.0 * n_hvp / t, trace_estimate=trace, status=st, per_probe=per_probe,
               nodes=[nodes[p, :steps[p]].tolist() for p in range(probes)],
               weights=[weights[p, :steps[p]].tolist() for p in range(probes)],
               density_edges=edges.tolist(), density_mass=mass.tolist())

    if w["reorth"] != "full":
        # windowed or no reorthogonalisation: repeat probe 0 (the same seed, so the
        # same run) for its (alpha, beta) and flag the ghost copies among its Ritz
        # values (section 7, Cullum-Willoughby test)
        al, be, s0, _ = mod.lanczos(m, args.seed, o)
        th, tw, resid, copies, spurious, n_ghosts = fd.ritz_diagnostics(al[:s0], be[:s0])
        same = np.allclose(np.sort(th), np.sort(nodes[0, :steps[0]]), rtol=1e-12, atol=0.0)
        say(f"probe 0 again: {s0} steps, Ritz values {'identical to' if same else 'DIFFERENT from'} the SLQ run; "
            f"{n_ghosts} ghost copies (duplicates within clusters); {int(spurious.sum())} values pass the "
            f"Cullum-Willoughby spurious test, total Gauss weight {tw[spurious].sum():.3e}")
        out["ghosts_probe0"] = dict(n_ghosts=n_ghosts, spurious=th[spurious].tolist(),
                                    spurious_weight=float(tw[spurious].sum()), copies=copies.tolist(),
                                    resid=resid.tolist(), identical_to_slq=bool(same))

    if args.block_diagonal:
        v = mod.random_vector(SEED_GAUSS, "gaussian")   # a Gaussian unit direction, as section 6 draws it
        t0 = time.perf_counter()
        bd = mod.block_diagonal(v)
        torch.cuda.synchronize()
        say(f"block-diagonal proxy of a Gaussian unit direction: {time.perf_counter() - t0:.1f} s")
        for i, r in enumerate(bd):
            say(f"layer {i}: relative error {r[1]:.4f}, cosine {r[2]:.4f}, |(Hv)_b| {r[3]:.4e}")
        out["block_diagonal"] = [dict(layer=i, abs_diff=float(r[0]), rel_err=float(r[1]), cosine=float(r[2]),
                                      hv_block_norm=float(r[3])) for i, r in enumerate(bd)]
    if args.out:
        with open(args.out, "w") as f:
            json.dump(out, f)
        say(f"wrote {args.out}")
    return out


if __name__ == "__main__":
    main()
