// lowp_cast.hpp -- device casts to the compute views of receivers below
// BF16 (App. D): FP8 E4M3 codes and MXFP4 blocks (E8M0 scale + E2M1 codes).
// Used by the dense cast, the lower-precision encode and the sparsifier's gate.
//
// Both casts run on gfx950's conversion unit.  Its behaviour at the edges,
// checked value by value against the CPU definitions (every FP32 pattern for
// FP8; every scaled value |q| < 8 and infinity for E2M1):
//   * v_cvt_pk_fp8_f32 gives OCP E4M3 with round-to-nearest-even, subnormal
//     results and signed zeros, but turns magnitudes that round above 448
//     (and infinity) into NaN, and every NaN into 0xFF.  Magnitudes are
//     therefore clamped to 448 first (448 is its own code, and the definition
//     saturates everything above it to 448), and NaN lanes are patched to
//     0x7F with their sign afterwards.
//   * v_cvt_scalef32_pk_fp4_f32 with scale 1 gives E2M1 with
//     round-to-nearest-even, saturation to +-6 (infinity included) and signed
//     zeros.  The block scale is applied before it, as an exact multiply by
//     2^-E.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pulse {

// y with its magnitude clamped to 448 and its sign kept; a NaN comes back as
// some value whose code is patched by the caller.
__device__ __forceinline__ float fp8_clamp(float y) {
  return __builtin_copysignf(__builtin_fminf(__builtin_fabsf(y), 448.0f), y);
}

// FP8 E4M3 codes of eight values, y[i] -> byte (i & 3) of lo (i < 4) or hi:
// nearest value, ties to the even code; |y| >= 448 and +-inf saturate to
// +-448; NaN -> 0x7F with y's sign; the sign of a zero result is kept.
// The NaN test is wave-wide (ballots of pairwise unordered compares), so
// the patch runs only in a wave that holds a NaN.
__device__ __forceinline__ void fp8_codes8(const float (&y)[8], uint32_t& lo, uint32_t& hi) {
  // the first conversion of each word writes bytes 0-1; bytes 2-3 of its
  // other input are overwritten by the second
  const float c1 = fp8_clamp(y[1]), c5 = fp8_clamp(y[5]);
  int a = __builtin_amdgcn_cvt_pk_fp8_f32(fp8_clamp(y[0]), c1, __float_as_int(c1), false);
  a = __builtin_amdgcn_cvt_pk_fp8_f32(fp8_clamp(y[2]), fp8_clamp(y[3]), a, true);
  int b = __builtin_amdgcn_cvt_pk_fp8_f32(fp8_clamp(y[4]), c5, __float_as_int(c5), false);
  b = __builtin_amdgcn_cvt_pk_fp8_f32(fp8_clamp(y[6]), fp8_clamp(y[7]), b, true);
  lo = (uint32_t)a;
  hi = (uint32_t)b;
  const uint64_t nan = __builtin_amdgcn_ballot_w64(__builtin_isunordered(y[0], y[1])) |
                       __builtin_amdgcn_ballot_w64(__builtin_isunordered(y[2], y[3])) |
                       __builtin_amdgcn_ballot_w64(__builtin_isunordered(y[4], y[5])) |
                       __builtin_amdgcn_ballot_w64(__builtin_isunordered(y[6], y[7]));
  if (nan) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (__builtin_isnan(y[i])) {
        const uint32_t c = 0x7Fu | ((__float_as_uint(y[i]) >> 24) & 0x80u);
        const int sh = 8 * (i & 3);
        uint32_t& w = i < 4 ? lo : hi;
        w = (w & ~(0xFFu << sh)) | (c << sh);
      }
    }
  }
}

// Bytes / nibbles of d that are nonzero, flagged in their top bit.
__device__ __forceinline__ uint32_t nonzero_bytes(uint32_t d) {
  return (((d & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | d) & 0x80808080u;
}
__device__ __forceinline__ uint32_t nonzero_nibbles(uint32_t d) {
  return (((d & 0x77777777u) + 0x77777777u) | d) & 0x88888888u;
}

// Eight flags at bits 4k (k = 0..7) moved to bits k.
__device__ __forceinline__ uint32_t gather_nibble_flags(uint32_t x) {
  x = (x | (x >> 3)) & 0x03030303u;
  x = (x | (x >> 6)) & 0x000F000Fu;
  return (x | (x >> 12)) & 0xFFu;
}

// Bit i set where the FP8 codes (lo, hi) and (olo, ohi) of value i differ.
__device__ __forceinline__ uint32_t fp8_change_mask(uint32_t lo, uint32_t hi, uint32_t olo,
                                                    uint32_t ohi) {
  const uint32_t d0 = lo ^ olo, d1 = hi ^ ohi;
  // even values' bytes, then odd values' bytes
  const uint32_t ev = __builtin_amdgcn_perm(d1, d0, 0x06040200u);
  const uint32_t od = __builtin_amdgcn_perm(d1, d0, 0x07050301u);
  return gather_nibble_flags((nonzero_bytes(ev) >> 7) | (nonzero_bytes(od) >> 3));
}

// Bit i set where nibble i of the packed E2M1 codes a and b differs.
__device__ __forceinline__ uint32_t nibble_change_mask(uint32_t a, uint32_t b) {
  return gather_nibble_flags(nonzero_nibbles(a ^ b) >> 3);
}

// MXFP4 view of 8 values held by one lane; the 4 lanes of a block (lane
// groups aligned to 4, all active) reduce their largest magnitude together.
// Returns the scale byte E + 127 with E = clamp(exponent field of the
// largest magnitude - 129, -127, 127), or 0xFF for a block holding a NaN;
// `packed` gets value i's E2M1 code in nibble i (all zero for a NaN block).
__device__ __forceinline__ uint32_t mx_view8(const float (&x)[8], uint32_t& packed) {
  uint32_t a[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = __float_as_uint(x[i]) & 0x7FFFFFFFu;
  const uint32_t m01 = a[0] > a[1] ? a[0] : a[1];
  const uint32_t m23 = a[2] > a[3] ? a[2] : a[3];
  const uint32_t m45 = a[4] > a[5] ? a[4] : a[5];
  const uint32_t m67 = a[6] > a[7] ? a[6] : a[7];
  const uint32_t m03 = m01 > m23 ? m01 : m23;
  const uint32_t m47 = m45 > m67 ? m45 : m67;
  uint32_t m = m03 > m47 ? m03 : m47;
  uint32_t o = (uint32_t)__builtin_amdgcn_update_dpp((int)m, (int)m, 0xB1, 0xF, 0xF, false);
  m = o > m ? o : m;  // lanes 4b .. 4b + 1 and 4b + 2 .. 4b + 3 pairwise (quad_perm 1,0,3,2)
  o = (uint32_t)__builtin_amdgcn_update_dpp((int)m, (int)m, 0x4E, 0xF, 0xF, false);
  m = o > m ? o : m;  // the two pairs (quad_perm 2,3,0,1)
  const bool nan = m > 0x7F800000u;
  // E + 127 = max(field - 2, 0); the field is at most 255 here, so E <= 126
  const int f2 = (int)(m >> 23) - 2;
  const uint32_t sc = (uint32_t)(f2 > 0 ? f2 : 0);
  const float inv = __uint_as_float((254u - sc) << 23);  // 2^-E, a normal number
  uint32_t p = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, x[0] * inv, x[1] * inv, 1.0f, 0);
  p = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p, x[2] * inv, x[3] * inv, 1.0f, 1);
  p = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p, x[4] * inv, x[5] * inv, 1.0f, 2);
  p = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p, x[6] * inv, x[7] * inv, 1.0f, 3);
  packed = nan ? 0u : p;
  return nan ? 0xFFu : sc;
}

}  // namespace pulse
