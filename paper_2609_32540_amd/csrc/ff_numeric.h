// Rounding helpers shared by the elementwise kernels of libff (device code).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ff {

typedef float ff_f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 ff_bf16x2 __attribute__((ext_vector_type(2)));

__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// two floats to a packed bf16 pair, nearest even (v_cvt_pk_bf16_f32)
__device__ inline uint32_t pack_bf16_rne(float a, float b) {
  ff_f32x2 f = {a, b};
  ff_bf16x2 h = __builtin_convertvector(f, ff_bf16x2);
  return __builtin_bit_cast(uint32_t, h);
}

// float64 -> float32 rounded to odd: truncate toward zero and set the last
// bit when inexact.  Rounding that result to bf16 (8 significant bits, far
// fewer than float32's 24) to nearest even equals rounding x directly.
__device__ inline float round_to_odd_f32(double x) {
  const float r = float(x);  // nearest even
  const double rd = double(r);
  if (rd == x) return r;
  uint32_t bits = __float_as_uint(r);
  if (fabs(rd) > fabs(x)) bits -= 1;  // one step toward zero
  return __uint_as_float(bits | 1u);
}

}  // namespace ff
