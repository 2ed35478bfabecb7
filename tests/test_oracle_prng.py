"""Pins of the oracle's integer streams and sample schedule (CPU only)."""
import os

import numpy as np
import pytest

from oracle import prng


def _vectors(golden_dir):
    out = {"splitmix64": [], "fmix32": []}
    with open(os.path.join(golden_dir, "prng_vectors.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            name, *vals = line.split()
            out[name].append([int(v, 0) for v in vals])
    return out


def test_splitmix64_published_vectors(golden_dir):
    for state, *expect in _vectors(golden_dir)["splitmix64"]:
        s = prng.SplitMix64(state)
        assert [s.next() for _ in expect] == expect


def test_fmix32_published_vectors(golden_dir):
    for x, expect in _vectors(golden_dir)["fmix32"]:
        assert prng.fmix32(x) == expect
        assert int(prng.fmix32(np.array([x], np.uint32))[0]) == expect


def test_below_range_and_rejection():
    s = prng.SplitMix64(123)
    for m in (1, 2, 3, 7, 1000, (1 << 63) + 5):
        for _ in range(50):
            v = s.below(m)
            assert 0 <= v < m
    # m = 2^63 + 5: the top 2^63 - 5 outputs are rejected; the returned value is
    # r mod m of the first accepted draw.
    m = (1 << 63) + 5
    s1, s2 = prng.SplitMix64(7), prng.SplitMix64(7)
    v = s1.below(m)
    while True:
        r = s2.next()
        if r < (1 << 64) - ((1 << 64) % m):
            break
    assert v == r % m


def test_below_is_uniform_on_small_m():
    s = prng.SplitMix64(99)
    counts = np.bincount([s.below(6) for _ in range(60000)], minlength=6)
    assert np.all(np.abs(counts - 10000) < 5 * np.sqrt(10000))


def test_derive_key_separates_inputs():
    keys = {prng.derive_key(0, t, a, b, c) for t in (1, 2) for a in range(4)
            for b in range(4) for c in range(4)}
    assert len(keys) == 2 * 64


@pytest.mark.parametrize("h", [1, 2, 3, 4, 5, 6])
def test_feistel_is_bijection_exhaustive(h):
    keys = prng.round_keys(5, 3, 11)
    x = np.arange(1 << (2 * h), dtype=np.uint32)
    y = prng.feistel(x, keys, h)
    assert np.array_equal(np.sort(y), x)


def test_half_bits():
    assert [prng.half_bits(S) for S in (0, 1, 2, 3, 4, 5, 16, 17, 1024, 1025, 20480, 65536)] == \
        [0, 0, 1, 1, 1, 2, 2, 3, 5, 6, 8, 8]


@pytest.mark.parametrize("S", [0, 1, 2, 3, 5, 16, 17, 100, 1024, 8192, 20480, 65537])
def test_schedule_is_permutation(S):
    for worker, rnd in ((0, 0), (3, 7)):
        p = prng.schedule(S, 0, worker, rnd)
        assert p.dtype == np.int32 and p.shape == (S,)
        assert np.array_equal(np.sort(p), np.arange(S))


def test_schedule_depends_on_worker_round_seed():
    a = prng.schedule(1024, 0, 0, 0)
    assert not np.array_equal(a, prng.schedule(1024, 0, 1, 0))
    assert not np.array_equal(a, prng.schedule(1024, 0, 0, 1))
    assert not np.array_equal(a, prng.schedule(1024, 1, 0, 0))
    assert np.array_equal(a, prng.schedule(1024, 0, 0, 0))


def test_schedule_cycle_walk_matches_scalar_walk():
    # Brute-force scalar restatement of the cycle walk on a non-power-of-4 S.
    S, h = 37, prng.half_bits(37)
    keys = prng.round_keys(2, 1, 4)
    expect = []
    for p in range(S):
        x = int(prng.feistel(np.array([p], np.uint32), keys, h)[0])
        while x >= S:
            x = int(prng.feistel(np.array([x], np.uint32), keys, h)[0])
        expect.append(x)
    assert prng.schedule(S, 2, 1, 4).tolist() == expect
