// fp8.hpp - the 8-bit E4M3 KV-cache code on gfx950: quantisation of a float
// (in software, exact) and conversion of stored codes to bf16 for the
// matrix cores (the native conversion instruction).
// Internal to libsq.
//
// E4M3 (the OCP 8-bit format, gfx950's native FP8): sign, 4 exponent bits
// with bias 7, 3 mantissa bits; exponent field 0 holds the subnormals
// m * 2^-9; codes 0x7F / 0xFF are NaN; the largest finite magnitude is 448.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace sq {

// The code nearest to y (ties to the even code), magnitudes >= 448
// saturating to 448, the sign of y kept.  y must not be NaN.
__device__ inline uint32_t e4m3_encode(float y) {
  const uint32_t u = __float_as_uint(y);
  const uint32_t sign = (u >> 24) & 0x80u;
  const float a = __uint_as_float(u & 0x7fffffffu);
  uint32_t code;
  if (a >= 448.f) {
    code = 0x7eu;
  } else {
    const int e = (int)((u >> 23) & 0xffu) - 127;
    if (e >= -6) { // normal: round the 23-bit mantissa to 3 bits
      const uint32_t m23 = u & 0x7fffffu;
      uint32_t m3 = m23 >> 20;
      const uint32_t rem = m23 & 0xfffffu;
      m3 += (rem > 0x80000u || (rem == 0x80000u && (m3 & 1u))) ? 1u : 0u;
      code = ((uint32_t)(e + 7) << 3) + m3; // m3 == 8 carries into the exponent
    } else { // subnormal steps of 2^-9 (the product is exact; rint rounds to even)
      code = (uint32_t)__builtin_rintf(a * 512.f);
    }
  }
  return code | sign;
}

// Four codes (bytes of w, lowest first) as four bf16 values (two 32-bit
// words, lowest first).  Exact for every finite code.
__device__ inline uint2 e4m3x4_to_bf16(uint32_t w) {
  const auto lo = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, false);
  const auto hi = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, true);
  return make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
}

} // namespace sq
