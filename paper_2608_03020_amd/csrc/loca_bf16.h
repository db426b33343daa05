// loca_bf16.h -- packed float -> bf16 conversions and the three-part bf16 split.
//
// Both use the hardware's v_cvt_pk_bf16_f32 (round to nearest even) two values at a time;
// a packed part is turned back into floats by a shift (low half) or a mask (high half), so
// a value costs one conversion per part and no repacking.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace loca {

typedef float f32x2_v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));

// (a, b) as a packed bf16 pair, a in the low half
__device__ __forceinline__ uint32_t cvt_pk_bf16(float a, float b) {
  const f32x2_v v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_v));
}
__device__ __forceinline__ float bf16_lo(uint32_t p) { return __uint_as_float(p << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t p) { return __uint_as_float(p & 0xffff0000u); }

// a = h + m + l for a pair of floats (each part packed as above): h = bf16(a),
// m = bf16(a - h), l = bf16(a - h - m); the differences are exact in float, and the parts
// hold a to about 2^-27 relative.
__device__ __forceinline__ void split3_pair(float a0, float a1, uint32_t& hp, uint32_t& mp, uint32_t& lp) {
  hp = cvt_pk_bf16(a0, a1);
  const float r0 = a0 - bf16_lo(hp), r1 = a1 - bf16_hi(hp);
  mp = cvt_pk_bf16(r0, r1);
  const float s0 = r0 - bf16_lo(mp), s1 = r1 - bf16_hi(mp);
  lp = cvt_pk_bf16(s0, s1);
}

}  // namespace loca
