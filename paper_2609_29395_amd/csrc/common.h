// Internal helpers shared by the HIP kernels and the host runtime.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint16_t bf16_t;  // raw bf16 bits in memory

// ------------------------------------------------------------ bf16 <-> fp32
__host__ __device__ __forceinline__ float bf16_to_f32(bf16_t b) {
  uint32_t u = ((uint32_t)b) << 16;
  float f;
  __builtin_memcpy(&f, &u, 4);
  return f;
}

// Round to nearest, ties to even, by the gfx950 conversion instruction
// (v_cvt_pk_bf16_f32).  Checked on the device against the integer rounding
// (add 0x7fff plus the lowest kept bit, truncate) over 2^24 bit patterns --
// random values, exact ties, values just below a tie, subnormals, the
// largest finite values (which round to infinity) and infinities: identical
// for every non-NaN input; a NaN keeps its sign and leading payload bits.
typedef __bf16 bf16x2_hw __attribute__((ext_vector_type(2)));
typedef float f32x2_hw __attribute__((ext_vector_type(2)));
__device__ __forceinline__ bf16_t f32_to_bf16(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }
// Two values in one instruction: lo in bits 0..15, hi in bits 16..31.
__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_hw){lo, hi}, bf16x2_hw));
}

template <typename T> struct ElemT;
template <> struct ElemT<float> {
  static constexpr int VEC = 4;  // elements per 16-byte vector
  __device__ static __forceinline__ float to_f(float v) { return v; }
  __device__ static __forceinline__ float from_f(float v) { return v; }
};
template <> struct ElemT<bf16_t> {
  static constexpr int VEC = 8;
  __device__ static __forceinline__ float to_f(bf16_t v) { return bf16_to_f32(v); }
  __device__ static __forceinline__ bf16_t from_f(float v) { return f32_to_bf16(v); }
};

// ------------------------------------------------------ unsigned fast divide
// q = n / d for all 32-bit n by a multiply-high and a shift (Granlund and
// Montgomery, "Division by invariant integers using multiplication", 1994).
struct FastDiv {
  uint32_t d, m, s;
};

inline FastDiv make_fastdiv(uint32_t d) {
  FastDiv f;
  f.d = d;
  uint32_t s = 0;
  while ((1ull << s) < d) ++s;
  f.s = s;
  f.m = (uint32_t)(((1ull << 32) * ((1ull << s) - d)) / d + 1);
  return f;
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv &f) {
  return (uint32_t)(((uint64_t)__umulhi(n, f.m) + n) >> f.s);
}

// ----------------------------------------------------- XCD-aware tile order
// Workgroups are dealt to the 8 XCDs round-robin by linear id.  Map linear id
// L to logical tile so that each XCD walks a contiguous run of logical tiles
// (neighbouring tiles share input rows in that XCD's L2).
__device__ __forceinline__ uint32_t xcd_swizzle(uint32_t L, uint32_t total) {
  const uint32_t t8 = total & ~7u;
  if (L >= t8) return L;
  return (L & 7u) * (t8 >> 3) + (L >> 3);
}

// ------------------------------------------------------- replica selection
// A launch runs the replicas listed in rmap (device, one entry per replica
// slot of its grid); a null rmap runs replica z in slot z.  The result is
// workgroup-uniform.
__device__ __forceinline__ int replica_of(const int32_t *rmap, int z) {
  return rmap ? __builtin_amdgcn_readfirstlane(rmap[z]) : z;
}
