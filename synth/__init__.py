"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This module is an input generator only: it holds none of the arithmetic of the
finite-difference Hessian-vector product, Lanczos or quadrature.  It draws

* parameter vectors (N(0, 0.02) matrices, unit gains, zero biases), given a list
  of ranges that the caller takes from its own parameter layout;
* token batches, uniform over the vocabulary or Zipf(s) distributed, standing in
  for the natural-language corpora the paper measures on (wikitext-2, the Pile);
* Rademacher probes z/sqrt(P) and Gaussian directions.

Every draw comes from one counter-based generator, SplitMix64 (Steele, Lea and
Flood, "Fast splittable pseudorandom number generators", OOPSLA 2014), used in
its counter form: the i-th output (0-based) of the stream with 64-bit state
``key`` is ``mix(key + (i + 1) * GAMMA) mod 2**64``.  The key of a (seed, stream)
pair is ``seed * 2**16 + stream``.  The GPU library implements the same
published generator on its own; this is the CPU side's implementation.

Derived variates (all computed in float64, exactly reproducible from integers):

* uniform   u = ((h >> 11) + 0.5) * 2**-53, strictly inside (0, 1);
* normal    Box-Muller, cosine branch only: element i uses outputs 2i and 2i+1,
            n = sqrt(-2 ln u(2i)) * cos(2 pi u(2i+1));
* sign      -1 if the top bit of output i is set, else +1;
* uniform token   ((h >> 32) * V) >> 32 (integer multiply-high, no modulo bias);
* Zipf token      inverse CDF: the smallest rank k (1-based) with
                  cdf[k] >= u, where cdf[k] = sum_{j<=k} j**-s / sum_{j<=V} j**-s,
                  mapped to token id k - 1.
"""
from __future__ import annotations

import concurrent.futures as cf
import os

import numpy as np

GAMMA = np.uint64(0x9E3779B97F4A7C15)
_C1 = np.uint64(0xBF58476D1CE4E5B9)
_C2 = np.uint64(0x94D049BB133111EB)

# Stream numbers: one per purpose, so draws for different purposes never overlap.
STREAM_PARAMS = 1
STREAM_TOKENS = 2
STREAM_PROBE = 3
STREAM_GAUSS = 4

# Parameter kinds in a layout range list.
KIND_MATRIX = 0   # N(0, std) entries
KIND_GAIN = 1     # ones
KIND_BIAS = 2     # zeros

_CHUNK = 1 << 22


def _key(seed: int, stream: int) -> np.uint64:
    return np.uint64(((int(seed) << 16) + int(stream)) & 0xFFFFFFFFFFFFFFFF)


def _mix(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * _C1
    z = (z ^ (z >> np.uint64(27))) * _C2
    return z ^ (z >> np.uint64(31))


def splitmix64(seed: int, stream: int, index) -> np.ndarray:
    """Outputs number ``index`` (uint64 array or scalar) of stream (seed, stream)."""
    idx = np.asarray(index, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = _key(seed, stream) + (idx + np.uint64(1)) * GAMMA
        return _mix(z)


def splitmix64_state(state: int, n: int) -> np.ndarray:
    """First n outputs of the plain sequential generator started at ``state``."""
    idx = np.arange(n, dtype=np.uint64)
    with np.errstate(over="ignore"):
        return _mix(np.uint64(state) + (idx + np.uint64(1)) * GAMMA)


def uniform(seed: int, stream: int, index) -> np.ndarray:
    h = splitmix64(seed, stream, index)
    return ((h >> np.uint64(11)).astype(np.float64) + 0.5) * (2.0 ** -53)


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _chunked(fn, n: int, out: np.ndarray) -> np.ndarray:
    """Fill out[c0:c1] = fn(c0, c1) over chunks of _CHUNK elements on a thread
    pool (numpy releases the GIL inside these element-wise kernels); every
    element depends on its own index only, so the result does not depend on
    the chunking or the thread count."""
    bounds = [(c0, min(n, c0 + _CHUNK)) for c0 in range(0, n, _CHUNK)]
    if len(bounds) <= 1:
        for c0, c1 in bounds:
            out[c0:c1] = fn(c0, c1)
        return out

    def work(b):
        out[b[0]:b[1]] = fn(b[0], b[1])

    with cf.ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(work, bounds))
    return out


def normal(seed: int, stream: int, start: int, n: int) -> np.ndarray:
    """Standard normals for elements start .. start+n-1 of (seed, stream)."""
    def fn(c0, c1):
        i = np.arange(start + c0, start + c1, dtype=np.uint64)
        u1 = uniform(seed, stream, i * np.uint64(2))
        u2 = uniform(seed, stream, i * np.uint64(2) + np.uint64(1))
        return np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * np.pi * u2)
    return _chunked(fn, n, np.empty(n, dtype=np.float64))


def rademacher(seed: int, n: int, stream: int = STREAM_PROBE) -> np.ndarray:
    """Signs in {-1, +1} as float64, element i from output i."""
    def fn(c0, c1):
        h = splitmix64(seed, stream, np.arange(c0, c1, dtype=np.uint64))
        return np.where((h >> np.uint64(63)) == np.uint64(1), -1.0, 1.0)
    return _chunked(fn, n, np.empty(n, dtype=np.float64))


def rademacher_probe(seed: int, n: int) -> np.ndarray:
    """Unit-norm probe z / sqrt(n) rounded to float32 (the stored probe)."""
    return (rademacher(seed, n) / np.sqrt(float(n))).astype(np.float32)


def gaussian_direction(seed: int, n: int) -> np.ndarray:
    """v ~ N(0, I) normalised to unit length, float64."""
    g = normal(seed, STREAM_GAUSS, 0, n)
    return g / np.linalg.norm(g)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 by round-to-nearest-even, returned as float32 values."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    r = ((b + np.uint32(0x7FFF) + lsb) & np.uint32(0xFFFF0000)).astype(np.uint32)
    return r.view(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) of float32 values that are bf16-exact."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return (b >> np.uint32(16)).astype(np.uint16)


def init_params(ranges, n_params: int, seed: int, std: float = 0.02,
                bf16: bool = False) -> np.ndarray:
    """Flat parameter vector (float32 values; bf16-exact when ``bf16``).

    ``ranges`` is a list of (offset, numel, kind).  A matrix entry at flat index
    i is float32(std * normal(seed, STREAM_PARAMS, i)); gains are 1, biases 0.
    """
    theta = np.zeros(n_params, dtype=np.float32)
    for off, numel, kind in ranges:
        if kind == KIND_MATRIX:
            theta[off:off + numel] = (std * normal(seed, STREAM_PARAMS, off, numel)).astype(np.float32)
        elif kind == KIND_GAIN:
            theta[off:off + numel] = 1.0
        elif kind == KIND_BIAS:
            theta[off:off + numel] = 0.0
        else:
            raise ValueError(f"unknown parameter kind {kind}")
    if bf16:
        theta = bf16_round(theta)
    return theta


def zipf_cdf(vocab: int, s: float = 1.1) -> np.ndarray:
    w = np.arange(1, vocab + 1, dtype=np.float64) ** (-s)
    c = np.cumsum(w)
    return c / c[-1]


def tokens(seed: int, batch: int, seq: int, vocab: int, dist: str = "uniform",
           s: float = 1.1) -> np.ndarray:
    """int32 [batch, seq] token ids; element t = b*seq + s uses output t."""
    n = batch * seq
    idx = np.arange(n, dtype=np.uint64)
    if dist == "uniform":
        h = splitmix64(seed, STREAM_TOKENS, idx)
        tok = ((h >> np.uint64(32)) * np.uint64(vocab)) >> np.uint64(32)
        out = tok.astype(np.int64)
    elif dist == "zipf":
        u = uniform(seed, STREAM_TOKENS, idx)
        cdf = zipf_cdf(vocab, s)
        out = np.searchsorted(cdf, u, side="left").astype(np.int64)
        out = np.minimum(out, vocab - 1)
    else:
        raise ValueError(dist)
    return out.reshape(batch, seq).astype(np.int32)
