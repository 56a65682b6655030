// Internal helpers shared by the LLEP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "llep.h"

namespace llep {

constexpr int kWave = 64;
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ uint64_t lanemask_lt() {
  return (uint64_t(1) << lane_id()) - 1;
}

// Mask of the active lanes holding the same value v (v < 2^nbits), built
// from one ballot per bit. Every lane of the wave must be active.
__device__ __forceinline__ uint64_t match_any(uint32_t v, int nbits) {
  uint64_t m = __ballot(1);
  for (int b = 0; b < nbits; ++b) {
    const uint32_t bit = (v >> b) & 1u;
    const uint64_t on = __ballot(bit);
    m &= bit ? on : ~on;
  }
  return m;
}

// Bits needed to hold values 0 .. v.
__host__ __device__ inline int bits_for(uint32_t v) {
  int n = 1;
  while ((v >> n) != 0) ++n;
  return n;
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(uint32_t(h) << 16);
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two floats -> a packed bfloat16 pair (lo in bits 0..15), rounded to
// nearest even (NaN stays NaN) by the gfx950 pair conversion
// (v_cvt_pk_bf16_f32: one instruction, no branch). For every input that is
// not a NaN it gives the bits of the rounding formula
// (u + 0x7fff + ((u >> 16) & 1)) >> 16 on the float's bits u.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// float -> bfloat16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return uint16_t(pack_bf16x2(f, 0.0f));
}

}  // namespace llep
