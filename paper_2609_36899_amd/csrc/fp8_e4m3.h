// OCP 8-bit E4M3FN encoding of KV values, shared by the device kernels that
// write fp8 pages and the host library (which exports it for bit-exact
// checks on the CPU).
//
// Format: sign, 4 exponent bits (bias 7), 3 mantissa bits; subnormals
// m * 2^-9; largest finite 448; S.1111.111 is NaN (never produced here).
// Round to nearest, ties to even, saturating at +-448; the sign is kept on
// values that round to zero.  Exact integer steps on the float's bits.
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define PDEC_HD __host__ __device__
#else
#include <math.h>
#define PDEC_HD
#endif

namespace pdec {

PDEC_HD inline uint32_t e4m3_from_f32(float x) {
  const uint32_t b = __builtin_bit_cast(uint32_t, x);
  const uint32_t sign = (b >> 24) & 0x80u;
  const float a = fabsf(x);
  if (!(a < 448.f)) return sign | 0x7Eu;  // saturate (NaN inputs too)
  // Subnormal step 2^-9: a * 512 is exact, and rintf rounds it to nearest
  // even (the default rounding mode on both sides); 8 rounds to 0x08, the
  // smallest normal code.
  if (a < 0x1p-6f) return sign | (uint32_t)rintf(a * 512.f);
  const uint32_t mant = b & 0x7FFFFFu;
  const uint32_t r = mant + 0x7FFFFu + ((mant >> 20) & 1u);  // RNE to 3 mantissa bits
  const int e = (int)((b >> 23) & 0xFFu) - 127 + (int)(r >> 23);
  return sign | ((uint32_t)(e + 7) << 3) | ((r >> 20) & 7u);
}

}  // namespace pdec

#undef PDEC_HD
