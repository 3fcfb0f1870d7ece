"""Pins for the shared seeded input generator (CPU)."""
import os

import numpy as np
import pytest

import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "splitmix64.txt")


def test_splitmix64_published_vectors():
    rows = [l.split() for l in open(GOLDEN) if l.strip() and not l.startswith("#")]
    assert len(rows) == 8
    for state, idx, val in rows:
        out = synth.splitmix64_state(int(state), int(idx) + 1)
        assert int(out[int(idx)]) == int(val)


def test_counter_form_matches_key():
    # stream (seed, stream) is the sequential generator started at seed*2^16+stream
    seed, stream = 7, 3
    a = synth.splitmix64(seed, stream, np.arange(10, dtype=np.uint64))
    b = synth.splitmix64_state((seed << 16) + stream, 10)
    assert np.array_equal(a, b)


def test_uniform_open_interval_and_moments():
    u = synth.uniform(5, 1, np.arange(200000, dtype=np.uint64))
    assert u.min() > 0.0 and u.max() < 1.0
    assert abs(u.mean() - 0.5) < 5 * np.sqrt(1 / 12 / u.size)
    assert abs(u.var() - 1 / 12) < 0.002


def test_normal_moments():
    n = synth.normal(11, synth.STREAM_PARAMS, 0, 400000)
    se = 1 / np.sqrt(n.size)
    assert abs(n.mean()) < 5 * se
    assert abs(n.var() - 1.0) < 5 * np.sqrt(2) * se
    # fourth moment of N(0,1) is 3
    assert abs((n ** 4).mean() - 3.0) < 0.06
    # offset slices agree with the full draw
    assert np.array_equal(synth.normal(11, 1, 1234, 100), n[1234:1334])


def test_rademacher_probe():
    z = synth.rademacher(9, 100000)
    assert set(np.unique(z)) == {-1.0, 1.0}
    assert abs(z.mean()) < 5 / np.sqrt(z.size)
    q = synth.rademacher_probe(9, 1000)
    assert q.dtype == np.float32
    assert abs(np.linalg.norm(q.astype(np.float64)) - 1.0) < 1e-6


def test_bf16_round_to_nearest_even():
    one = np.float32(1.0)
    ulp = 2.0 ** -7  # bf16 spacing at 1.0
    xs = np.array([1.0, 1.0 + ulp / 2, 1.0 + 1.5 * ulp, 1.0 + ulp / 2 + 2 ** -20, -3.0,
                   1.0 + ulp / 4], dtype=np.float32)
    got = synth.bf16_round(xs)
    want = np.array([1.0, 1.0, 1.0 + 2 * ulp, 1.0 + ulp, -3.0, 1.0], dtype=np.float32)
    assert np.array_equal(got, want)
    assert synth.bf16_bits(np.array([one]))[0] == 0x3F80


def test_uniform_tokens_cover_vocab():
    t = synth.tokens(2, 64, 64, 256, "uniform")
    assert t.dtype == np.int32 and t.shape == (64, 64)
    assert t.min() >= 0 and t.max() < 256
    counts = np.bincount(t.reshape(-1), minlength=256)
    expect = t.size / 256
    chi2 = ((counts - expect) ** 2 / expect).sum()
    assert chi2 < 256 + 6 * np.sqrt(2 * 256)


def test_zipf_tokens_follow_pmf():
    V, s = 50, 1.1
    t = synth.tokens(2, 200, 500, V, "zipf", s)
    counts = np.bincount(t.reshape(-1), minlength=V).astype(np.float64)
    pmf = np.arange(1, V + 1, dtype=np.float64) ** -s
    pmf /= pmf.sum()
    expect = pmf * t.size
    chi2 = ((counts - expect) ** 2 / expect).sum()
    assert chi2 < V + 6 * np.sqrt(2 * V)
    # rank 1 is the most frequent token id 0
    assert counts.argmax() == 0


def test_init_params_kinds():
    ranges = [(0, 1000, synth.KIND_MATRIX), (1000, 10, synth.KIND_GAIN), (1010, 5, synth.KIND_BIAS)]
    th = synth.init_params(ranges, 1015, seed=1)
    assert np.all(th[1000:1010] == 1.0) and np.all(th[1010:] == 0.0)
    assert abs(th[:1000].std() - 0.02) < 0.003
    # element i of a matrix depends only on its flat index
    th2 = synth.init_params([(500, 500, synth.KIND_MATRIX)], 1000, seed=1)
    assert np.array_equal(th2[500:], th[500:1000])
    tb = synth.init_params(ranges, 1015, seed=1, bf16=True)
    assert np.array_equal(tb, synth.bf16_round(th))
