// Device-side helpers shared by the gfx950 kernels of the MoL library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mol.h"

namespace mol {

// Kernel-side view of a mol_problem (plain pointers, P precomputed).
struct DevProb {
  int B, N, Pq, Px, P, d, H, dtype;
  unsigned flags;   // MOL_FLAG_* bits
  const void* Q;
  const void* X;
  const float* a_q;
  const float* a_x;
  const void* W1;
  const float* b1;
  const void* W2;
  const float* b2;
};

// bf16 values are carried as their uint16 bit patterns.
typedef uint16_t bf16_t;

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16_t v) {
  return __uint_as_float(static_cast<uint32_t>(v) << 16);
}

// ---------------------------------------------------------------------------
// Sort keys.  A (score, item) pair maps to one 64-bit key whose unsigned
// order is (score descending, item ascending) when keys are sorted
// descending: high word = order-preserving image of the float score,
// low word = bitwise NOT of the item index.  Key 0 is below every real key
// and marks an empty slot.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t float_to_ordered(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;                   // -0 sorts as +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float ordered_to_float(uint32_t o) {
  uint32_t u = (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o;
  return __uint_as_float(u);
}
__device__ __forceinline__ uint64_t make_key(float score, int32_t item) {
  return (static_cast<uint64_t>(float_to_ordered(score)) << 32) |
         static_cast<uint32_t>(~static_cast<uint32_t>(item));
}
__device__ __forceinline__ float key_score(uint64_t key) {
  return key == 0 ? -__builtin_inff() : ordered_to_float(static_cast<uint32_t>(key >> 32));
}
__device__ __forceinline__ int32_t key_item(uint64_t key) {
  return key == 0 ? -1 : static_cast<int32_t>(~static_cast<uint32_t>(key));
}

// Round a float64 value to bf16, nearest-even, returning the bit pattern.
__device__ __forceinline__ bf16_t f64_to_bf16_rne(double x) {
  uint64_t bits = static_cast<uint64_t>(__double_as_longlong(x));
  const uint64_t sign = (bits >> 63) & 1u;
  const uint64_t mag = bits & 0x7FFFFFFFFFFFFFFFull;
  if (mag == 0) return static_cast<bf16_t>(sign << 15);
  const int e = static_cast<int>(mag >> 52) - 1023;   // unbiased exponent
  if (e < -126) {
    // bf16 subnormal range: multiples of 2^-133.
    double q = rint(fabs(x) * 0x1p133);                // rint: ties to even
    return static_cast<bf16_t>((sign << 15) | static_cast<uint32_t>(q));
  }
  // keep 7 explicit mantissa bits: drop 45 bits with round-to-nearest-even
  const uint64_t lsb = (mag >> 45) & 1u;
  const uint64_t r = (mag + 0x00000FFFFFFFFFFFull + lsb) >> 45;   // exp11 | mant7
  const int e8 = static_cast<int>(r >> 7) - 1023 + 127;
  if (e8 >= 255) return static_cast<bf16_t>((sign << 15) | 0x7F80u);
  return static_cast<bf16_t>((sign << 15) | (static_cast<uint32_t>(e8) << 7) |
                             static_cast<uint32_t>(r & 0x7Fu));
}

}  // namespace mol
