// Integer random streams and the keyed permutation used for sampling.
//
// The paper fixes no generator.  Reading used here:
//  * SplitMix64 (Steele, Lea and Flood, 2014) and its mix64 finaliser;
//  * keys derived by chaining mix64 over (seed + tag, a, b) with additions
//    modulo 2^64;
//  * a 4-round balanced Feistel network on the smallest even-bit domain
//    2^(2h) >= n, with cycle walking into [0, n) (Black and Rogaway,
//    "Ciphers with arbitrary finite domains", 2002): round i maps (L, R) to
//    (R, L xor F_i(R)), F_i(R) = mix64(key xor ((i+1) << 32 | R)) mod 2^h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define GCPSL_TAG_ASSIGN 0x41535349474Eull
#define GCPSL_TAG_SAMPLE 0x53414D504C45ull
#define GCPSL_GOLDEN 0x9E3779B97F4A7C15ull

__host__ __device__ __forceinline__ uint64_t gc_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__host__ __device__ __forceinline__ uint64_t gc_sample_key(uint64_t seed, uint64_t cluster,
                                                           uint64_t epoch) {
  uint64_t h = gc_mix64(seed + GCPSL_TAG_SAMPLE);
  h = gc_mix64(h + cluster);
  return gc_mix64(h + epoch);
}

// Half width h of the Feistel domain 2^(2h) for a permutation of [0, n).
__host__ __device__ __forceinline__ int gc_half_bits(uint32_t n) {
  int bits = 0;
  while (bits < 32 && (1ull << bits) < (uint64_t)n) ++bits;
  if (bits < 1) bits = 1;
  return (bits + 1) >> 1;
}

__host__ __device__ __forceinline__ uint32_t gc_feistel_pass(uint32_t x, uint64_t key, int h) {
  const uint32_t mask = (uint32_t)((1ull << h) - 1);
  uint32_t l = x >> h, r = x & mask;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t f = (uint32_t)(gc_mix64(key ^ (((uint64_t)(i + 1) << 32) | r)) & mask);
    const uint32_t t = r;
    r = l ^ f;
    l = t;
  }
  return (uint32_t)(((uint64_t)l << h) | r);
}

// pi(p) for the keyed permutation of [0, n), p < n.  The walk stays on the
// cycle of p inside the permutation of [0, 2^(2h)), which returns to [0, n)
// within 2^(2h) passes; the loop bound is that cycle-length limit.
__host__ __device__ __forceinline__ uint32_t gc_permute(uint32_t p, uint32_t n, uint64_t key) {
  if (n <= 1) return 0;
  const int h = gc_half_bits(n);
  const uint64_t limit = 1ull << (2 * h);
  uint32_t x = p;
  for (uint64_t it = 0; it < limit; ++it) {
    x = gc_feistel_pass(x, key, h);
    if (x < n) return x;
  }
  return p;  // unreachable for p < n
}
