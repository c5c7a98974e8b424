// lowp_cast.hpp -- device casts to the compute views of receivers below
// BF16 (App. D): FP8 E4M3 codes and MXFP4 blocks (E8M0 scale + E2M1 codes).
// Used by the lower-precision encode and by the sparsifier's gate.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pulse {

// FP8 E4M3 code of y: nearest value, ties to the even code; |y| >= 448 and
// +-inf saturate to +-448; NaN -> 0x7F with y's sign; the sign of a zero
// result is kept.  Normal results round the FP32 mantissa to 3 bits (a carry
// moves into the exponent); results below 2^-6 are multiples of 2^-9.
__device__ __forceinline__ uint32_t fp8_code(float y) {
  const uint32_t u = __float_as_uint(y);
  const uint32_t s = (u >> 24) & 0x80u;
  const uint32_t a = u & 0x7FFFFFFFu;
  if (a > 0x7F800000u) return s | 0x7Fu;
  if (a >= 0x43E00000u) return s | 0x7Eu;  // 448
  if (a < 0x3C800000u)                      // 2^-6
    return s | (uint32_t)__builtin_rintf(__uint_as_float(a) * 512.0f);
  const uint32_t r = (a + 0x7FFFFu + ((a >> 20) & 1u)) >> 20;
  return s | (r - ((127u - 7u) << 3));
}

// E2M1 code of q = x / 2^E: the compares place |q| among the midpoints of the
// magnitudes 0, 0.5, 1, 1.5, 2, 3, 4, 6; at a midpoint the even code wins
// (>= where the upper neighbour's code is even, > where it is odd), above 6
// the code saturates; the sign bit is x's.
__device__ __forceinline__ uint32_t e2m1_code(float q) {
  const float a = fabsf(q);
  const uint32_t c = (uint32_t)(a > 0.25f) + (uint32_t)(a >= 0.75f) + (uint32_t)(a > 1.25f) +
                     (uint32_t)(a >= 1.75f) + (uint32_t)(a > 2.5f) + (uint32_t)(a >= 3.5f) +
                     (uint32_t)(a > 5.0f);
  return c | ((__float_as_uint(q) >> 28) & 8u);
}

// Scale exponent E of a block from the largest magnitude's bits (NaN handled
// by the caller): clamp(exponent field - 129, -127, 127).
__device__ __forceinline__ int mx_exponent(uint32_t amax_bits) {
  const int E = (int)(amax_bits >> 23) - 129;
  return E < -127 ? -127 : E;  // the field is at most 255, so E <= 126
}

// MXFP4 view of 8 values held by one lane; the 4 lanes of a block (lane
// groups aligned to 4) reduce their largest magnitude together.  Returns the
// scale byte; codes[i] gets each value's code.
__device__ __forceinline__ uint32_t mx_view8(const float (&x)[8], uint32_t (&codes)[8]) {
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t b = __float_as_uint(x[i]) & 0x7FFFFFFFu;
    m = b > m ? b : m;
  }
  uint32_t o = __shfl_xor(m, 1);
  m = o > m ? o : m;
  o = __shfl_xor(m, 2);
  m = o > m ? o : m;
  if (m > 0x7F800000u) {  // a NaN in the block
#pragma unroll
    for (int i = 0; i < 8; ++i) codes[i] = 0;
    return 0xFFu;
  }
  const int E = mx_exponent(m);
  const float inv = __uint_as_float((uint32_t)(127 - E) << 23);  // 2^-E, exact
#pragma unroll
  for (int i = 0; i < 8; ++i) codes[i] = e2m1_code(x[i] * inv);
  return (uint32_t)(E + 127);
}

}  // namespace pulse
