// Packed float -> bf16 conversion for the two-plane summaries formed on the fly (one
// v_cvt_pk_bf16_f32 per pair: round to nearest even, as the scalar conversion, for the
// finite values a summary holds).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mkv {

typedef float f32x2_cvt __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_cvt __attribute__((ext_vector_type(2)));

// (a, b) as two bf16 in one dword, a in the low half.
__device__ __forceinline__ uint32_t bf16_pair(float a, float b) {
  const f32x2_cvt v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_cvt));
}

// The hi / lo split of a pair: hi = RNE(x), lo = RNE(x - hi), each as a packed dword.
__device__ __forceinline__ void bf16_split_pair(float a, float b, uint32_t& hi, uint32_t& lo) {
  hi = bf16_pair(a, b);
  lo = bf16_pair(a - __uint_as_float(hi << 16), b - __uint_as_float(hi & 0xffff0000u));
}

}  // namespace mkv
