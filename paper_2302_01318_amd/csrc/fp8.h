// OCP FP8 E4M3 codes of weight-only FP8 models: 1 sign bit, 4 exponent bits
// (bias 7), 3 mantissa bits, subnormals, no infinities, largest finite 448.
#pragma once
#include "common.h"

namespace sps {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Nearest E4M3 code of x, ties to the even code; |x| >= 448 saturates to
// +-448 and the sign is kept (a negative x that rounds to zero gives -0).
// Integer arithmetic on the fp32 pattern of x; x must be finite.
__device__ __forceinline__ uint32_t e4m3_encode(float x) {
  const uint32_t b = __float_as_uint(x);
  const uint32_t sign = (b >> 24) & 0x80u;
  const uint32_t a = b & 0x7fffffffu;
  uint32_t code;
  if (a >= 0x43e00000u) {                    // |x| >= 448
    code = 0x7eu;
  } else if (a >= 0x3c800000u) {             // |x| >= 2^-6: normal, exponent field (a >> 23) - 120
    const uint32_t m = a & 0x7fffffu;
    const uint32_t keep = m >> 20, rem = m & 0xfffffu;
    const uint32_t up = rem > 0x80000u || (rem == 0x80000u && (keep & 1u));
    code = (((a >> 23) - 120u) << 3) + keep + up;     // a mantissa carry moves into the exponent
  } else {                                   // subnormal range: |x| / 2^-9 rounded to an integer 0..8
    const uint32_t e = a >> 23;
    const uint32_t S = e ? ((a & 0x7fffffu) | 0x800000u) : a;   // |x| = S 2^(max(e,1) - 150)
    const int shift = 141 - static_cast<int>(e ? e : 1u);        // |x| 2^9 = S 2^-shift, shift >= 21
    if (shift >= 25) {
      code = 0;                              // S < 2^24 <= half an output unit
    } else {
      const uint32_t q = S >> shift, rem = S & ((1u << shift) - 1u), half = 1u << (shift - 1);
      code = q + (rem > half || (rem == half && (q & 1u)) ? 1u : 0u);
    }
  }
  return code | sign;
}

// Sixteen codes (byte i of the vector is code i) to two bf16 fragments:
// codes 0-7 -> lo, 8-15 -> hi. Every E4M3 value is a bf16 value, so the
// conversion (v_cvt_scalef32_pk_bf16_fp8 with scale 1) is exact.
__device__ __forceinline__ bf16x8 e4m3x8_to_bf16(uint32_t w0, uint32_t w1) {
  const bf16x2 a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w0, 1.0f, false);
  const bf16x2 b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w0, 1.0f, true);
  const bf16x2 c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w1, 1.0f, false);
  const bf16x2 d = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w1, 1.0f, true);
  return bf16x8{a[0], a[1], b[0], b[1], c[0], c[1], d[0], d[1]};
}
__device__ __forceinline__ void e4m3x16_to_frags(const u32x4 v, Frag<bf16>& lo, Frag<bf16>& hi) {
  lo.v = e4m3x8_to_bf16(v.x, v.y);
  hi.v = e4m3x8_to_bf16(v.z, v.w);
}

}  // namespace sps
