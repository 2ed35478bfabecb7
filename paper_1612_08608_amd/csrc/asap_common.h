// asap_common.h -- integer streams and the sample schedule, host and device.
//
// The paper leaves the order in which a replica visits its data open (each
// replica trains on its own portion, Section 5).  This library fixes it as a
// keyed permutation that any thread can evaluate at any position without a
// sort: a balanced 4-round Feistel network on 2h bits (Luby-Rackoff) whose
// round function is MurmurHash3's 32-bit finaliser, walked along its cycle
// until the value falls inside [0, S) (Black & Rogaway 2002).  Round keys
// come from SplitMix64 (Steele, Lea, Flood 2014) finalisers folded over
// (seed, tag, worker, round, j).  The same code runs on the host (graph
// builder, asap_schedule) and inside the SGD kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define ASAP_HD __host__ __device__ __forceinline__

namespace asap {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kTagGraph = 1;
constexpr uint64_t kTagSched = 2;

ASAP_HD uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

ASAP_HD uint64_t derive_key(uint64_t seed, uint64_t tag, uint64_t a, uint64_t b, uint64_t c) {
  uint64_t h = mix64(seed + kGamma);
  h = mix64((h ^ tag) + kGamma);
  h = mix64((h ^ a) + kGamma);
  h = mix64((h ^ b) + kGamma);
  h = mix64((h ^ c) + kGamma);
  return h;
}

ASAP_HD uint32_t fmix32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x85EBCA6Bu;
  x ^= x >> 13;
  x *= 0xC2B2AE35u;
  x ^= x >> 16;
  return x;
}

// Keyed permutation of [0, S) for one (worker, round).
struct Perm {
  uint32_t k0, k1, k2, k3;
  uint32_t h;     // half width in bits
  uint32_t mask;  // (1 << h) - 1
  uint32_t S;
};

ASAP_HD Perm perm_make(uint64_t seed, int32_t worker, int64_t round, uint32_t S) {
  Perm p;
  uint32_t nbits = 0;
  while (nbits < 32 && (uint64_t(1) << nbits) < uint64_t(S)) ++nbits;
  p.h = S < 2 ? 0u : (nbits + 1) / 2;
  p.mask = (p.h == 0) ? 0u : ((1u << p.h) - 1u);
  p.S = S;
  const uint64_t w = uint64_t(int64_t(worker)), r = uint64_t(round);
  p.k0 = uint32_t(derive_key(seed, kTagSched, w, r, 0));
  p.k1 = uint32_t(derive_key(seed, kTagSched, w, r, 1));
  p.k2 = uint32_t(derive_key(seed, kTagSched, w, r, 2));
  p.k3 = uint32_t(derive_key(seed, kTagSched, w, r, 3));
  return p;
}

ASAP_HD uint32_t feistel(const Perm& p, uint32_t x) {
  uint32_t L = x >> p.h, R = x & p.mask, t;
  t = L ^ (fmix32(R ^ p.k0) & p.mask); L = R; R = t;
  t = L ^ (fmix32(R ^ p.k1) & p.mask); L = R; R = t;
  t = L ^ (fmix32(R ^ p.k2) & p.mask); L = R; R = t;
  t = L ^ (fmix32(R ^ p.k3) & p.mask); L = R; R = t;
  return (L << p.h) | R;
}

// Position -> sample index.  The walk stays on the cycle through `pos`,
// which contains at least one value (pos itself) inside [0, S).
ASAP_HD uint32_t perm_at(const Perm& p, uint32_t pos) {
  if (p.S < 2) return 0u;
  uint32_t x = feistel(p, pos);
  while (x >= p.S) x = feistel(p, x);
  return x;
}

}  // namespace asap
