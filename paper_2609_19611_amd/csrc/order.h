// Location order (Sec. 4, "Search Heuristic"): the host-built prefix of
// corner and boundary locations, and the seeded permutation the device
// applies to the rest.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "graph.h"

namespace dg {

// Corner locations of every op (later ops first) and the first and last
// output location, each once, in rank order (see order.cpp).
std::vector<int64_t> order_prefix(const GraphIR& g, int64_t block_threads, int64_t warp);

}  // namespace dg

// Keyed permutation pi of [0, n): a balanced four-round Feistel network on
// 2h bits (the smallest h with 4^h >= n), round keys the first four outputs
// of SplitMix64 seeded with the caller's seed, round function the SplitMix64
// output mix of (half ^ key) cut to h bits; values at or past n are
// encrypted again until they fall below n (cycle walking).  Its inverse
// decrypts the same way.
struct DgPermKey {
  uint64_t k[4];
  uint64_t mask;  // 2^h - 1
  int32_t h;
  int32_t pad;
  int64_t n;
};

inline DgPermKey dg_perm_key(int64_t n, uint64_t seed) {
  DgPermKey K;
  int h = 0;
  while (h < 31 && ((uint64_t)1 << (2 * h)) < (uint64_t)n) ++h;
  K.h = h;
  K.pad = 0;
  K.mask = ((uint64_t)1 << h) - 1;
  K.n = n;
  uint64_t s = seed;
  for (int r = 0; r < 4; ++r) {
    s += 0x9E3779B97F4A7C15ull;
    uint64_t z = s;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    K.k[r] = z ^ (z >> 31);
  }
  return K;
}

// SplitMix64's output mix (Steele, Lea and Flood, 2014).
__host__ __device__ inline uint64_t dg_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// The network and its inverse on 2h-bit values: round r maps the halves
// (L, R) to (R, L ^ F_r(R)).
__host__ __device__ inline uint64_t dg_feistel(uint64_t x, const DgPermKey& K) {
  uint64_t L = x >> K.h, R = x & K.mask;
  for (int r = 0; r < 4; ++r) {
    const uint64_t t = L ^ (dg_mix64(R ^ K.k[r]) & K.mask);
    L = R;
    R = t;
  }
  return (L << K.h) | R;
}

__host__ __device__ inline uint64_t dg_feistel_inv(uint64_t x, const DgPermKey& K) {
  uint64_t L = x >> K.h, R = x & K.mask;
  for (int r = 3; r >= 0; --r) {
    const uint64_t t = R ^ (dg_mix64(L ^ K.k[r]) & K.mask);
    R = L;
    L = t;
  }
  return (L << K.h) | R;
}

// pi(i) for i < n: the cycle through i holds i itself, so the walk ends.
__host__ __device__ inline int64_t dg_perm_at(uint64_t i, const DgPermKey& K) {
  uint64_t v = dg_feistel(i, K);
  while (v >= (uint64_t)K.n) v = dg_feistel(v, K);
  return (int64_t)v;
}

// The position of value v < n: walking the cycle backwards.
__host__ __device__ inline int64_t dg_perm_position(uint64_t v, const DgPermKey& K) {
  uint64_t i = dg_feistel_inv(v, K);
  while (i >= (uint64_t)K.n) i = dg_feistel_inv(i, K);
  return (int64_t)i;
}
