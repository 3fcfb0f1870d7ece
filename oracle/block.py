"""Block-diagonal hypothesis statistics (oracle; section 6, Exp I).

For a unit probe v, h = Hv.  For each block b (the parameters of transformer
layer b), v^(b) is v with everything outside block b set to zero (not
renormalised) and h_b = H v^(b).  Restricted to block b, the two products are
compared by the absolute difference ||h^(b) - h_b^(b)||, the relative error
(that over ||h^(b)||) and the cosine similarity; the tables report mean and
standard deviation (population, ddof = 0) over blocks.
"""
from __future__ import annotations

import numpy as np


def block_stats(h: np.ndarray, hb_list, blocks):
    """``blocks`` is a list of (start, stop); ``hb_list[b]`` = H v^(b)."""
    absd, rel, cos = [], [], []
    for (s, e), hb in zip(blocks, hb_list):
        a = np.asarray(h[s:e], dtype=np.float64)
        b = np.asarray(hb[s:e], dtype=np.float64)
        diff = np.linalg.norm(a - b)
        na, nb = np.linalg.norm(a), np.linalg.norm(b)
        absd.append(diff)
        rel.append(diff / na)
        cos.append(float(a @ b) / (na * nb))
    absd, rel, cos = map(np.array, (absd, rel, cos))
    return {
        "abs": absd, "rel": rel, "cos": cos,
        "abs_mean": absd.mean(), "abs_std": absd.std(),
        "rel_mean": rel.mean(), "rel_std": rel.std(),
        "cos_mean": cos.mean(), "cos_std": cos.std(),
        "blocks": len(blocks),
    }


def masked(v: np.ndarray, start: int, stop: int) -> np.ndarray:
    out = np.zeros_like(v)
    out[start:stop] = v[start:stop]
    return out


def run(hvp, v: np.ndarray, blocks):
    """h = Hv and the per-block masked products, then the statistics."""
    h = hvp(v)
    hb = [hvp(masked(v, s, e)) for s, e in blocks]
    return block_stats(h, hb, blocks), h, hb
