"""Integer-only pseudo-random streams and the per-round sample schedule (oracle).

The paper gives no sampling rule beyond each replica training on its own
portion of the data and communicating after a few examples (Section 5).  The
reading used here, which the HIP library implements independently, is:

* SplitMix64 (Steele, Lea, Flood, OOPSLA 2014): state += 0x9E3779B97F4A7C15,
  output = mix64(state), with mix64 the published finaliser
  z ^= z >> 30; z *= 0xBF58476D1CE4E5B9; z ^= z >> 27; z *= 0x94D049BB133111EB;
  z ^= z >> 31 (all mod 2^64).
* Derived keys: K(seed, tag, a, b, c) starts from h = mix64(seed + gamma) and
  folds each of tag, a, b, c in as h = mix64((h xor v) + gamma).
* below(m): draw r, reject while r >= 2^64 - (2^64 mod m), return r mod m.
* Sample schedule of worker i in round r over S samples: a keyed permutation
  of [0, S) built as a balanced 4-round Feistel network on 2h bits
  (Luby-Rackoff), h = ceil(ceil(log2 S) / 2), with round function
  F_j(x) = fmix32(x xor k_j) & (2^h - 1), where fmix32 is MurmurHash3's 32-bit
  finaliser and k_j = low 32 bits of K(seed, SCHED, i, r, j); values outside
  [0, S) are walked along the cycle until they land inside (Black & Rogaway,
  "Ciphers with arbitrary finite domains", 2002).  Minibatch k of the round is
  positions [kB, min((k+1)B, S)) of that permutation.

Pins: SplitMix64 and fmix32 against published test vectors; below(m) range and
rejection threshold; the Feistel map is a bijection (exhaustive on small
domains) and every schedule is a permutation.
"""
from __future__ import annotations

import numpy as np

MASK64 = (1 << 64) - 1
MASK32 = (1 << 32) - 1
GAMMA = 0x9E3779B97F4A7C15

TAG_GRAPH = 1
TAG_SCHED = 2


def mix64(z: int) -> int:
    """SplitMix64 output finaliser on a 64-bit integer."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def derive_key(seed: int, tag: int, a: int = 0, b: int = 0, c: int = 0) -> int:
    h = mix64((seed + GAMMA) & MASK64)
    for v in (tag, a, b, c):
        h = mix64(((h ^ (v & MASK64)) + GAMMA) & MASK64)
    return h


class SplitMix64:
    """Sequential SplitMix64 stream."""

    def __init__(self, state: int):
        self.state = state & MASK64

    def next(self) -> int:
        self.state = (self.state + GAMMA) & MASK64
        return mix64(self.state)

    def below(self, m: int) -> int:
        """Unbiased integer in [0, m) by rejection of the top partial block."""
        if m <= 0:
            raise ValueError("below(m) needs m >= 1")
        rem = (1 << 64) % m
        while True:
            r = self.next()
            if rem == 0 or r < (1 << 64) - rem:
                return r % m


def fmix32(x):
    """MurmurHash3 32-bit finaliser; works on Python ints and uint32 arrays."""
    if isinstance(x, np.ndarray):
        x = x.astype(np.uint32)
        x ^= x >> np.uint32(16)
        x *= np.uint32(0x85EBCA6B)
        x ^= x >> np.uint32(13)
        x *= np.uint32(0xC2B2AE35)
        x ^= x >> np.uint32(16)
        return x
    x &= MASK32
    x ^= x >> 16
    x = (x * 0x85EBCA6B) & MASK32
    x ^= x >> 13
    x = (x * 0xC2B2AE35) & MASK32
    return x ^ (x >> 16)


def half_bits(S: int) -> int:
    """h such that the Feistel domain 4^h is the smallest even power of 2 >= S."""
    if S < 2:
        return 0
    nbits = (S - 1).bit_length()        # smallest b with 2^b >= S
    return (nbits + 1) // 2


def round_keys(seed: int, worker: int, rnd: int):
    return [derive_key(seed, TAG_SCHED, worker, rnd, j) & MASK32 for j in range(4)]


def feistel(x: np.ndarray, keys, h: int) -> np.ndarray:
    """One application of the 4-round Feistel bijection on [0, 4^h)."""
    mask = np.uint32((1 << h) - 1)
    x = x.astype(np.uint32)
    L = x >> np.uint32(h)
    R = x & mask
    for k in keys:
        F = fmix32(R ^ np.uint32(k)) & mask
        L, R = R, L ^ F
    return (L << np.uint32(h)) | R


def schedule(S: int, seed: int, worker: int, rnd: int) -> np.ndarray:
    """pi_{worker, rnd}: int32 permutation of [0, S) (cycle-walking Feistel)."""
    if S < 0:
        raise ValueError("S must be >= 0")
    if S <= 1:
        return np.zeros(S, np.int32)
    h = half_bits(S)
    keys = round_keys(seed, worker, rnd)
    x = feistel(np.arange(S, dtype=np.uint32), keys, h)
    out = x.copy()
    pending = out >= S
    while pending.any():
        out[pending] = feistel(out[pending], keys, h)
        pending = out >= S
    return out.astype(np.int32)
