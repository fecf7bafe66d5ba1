// OCP FP8 E4M3 encoding of stored coefficients (cache type FDKV_BF16_E4M3).
//
// E4M3: sign, 4 exponent bits (bias 7), 3 mantissa bits; subnormals are
// multiples of 2^-9; the largest finite value is 448 (S.1111.110) and
// S.1111.111 is NaN (no infinities).  Encoding rounds to nearest, ties to
// even, and saturates everything beyond 448 to +-448.  Decoding is done by
// the gfx950 conversion instructions, which follow the same format.
//
// Plain C++ usable on the host, so the encoder can be checked on the CPU.
#pragma once
#include <stdint.h>
#include <string.h>

#if defined(__HIPCC__)
#define FDKV_F8_HD __host__ __device__ __forceinline__
#else
#include <math.h>
#define FDKV_F8_HD inline
#endif

namespace fdkv {

FDKV_F8_HD uint8_t f32_to_e4m3(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  const uint32_t sign = (u >> 24) & 0x80u;
  const uint32_t a = u & 0x7FFFFFFFu;
  if (a > 0x7F800000u) return (uint8_t)(sign | 0x7Fu);  // NaN
  uint32_t code;
  if (a >= 0x3C800000u) {                                // |x| >= 2^-6: normal
    const uint32_t e = (a >> 23) - 127u + 7u;            // biased E4M3 exponent, >= 1
    const uint32_t m = a & 0x7FFFFFu;
    const uint32_t r = (m + 0x7FFFFu + ((m >> 20) & 1u)) >> 20;  // 3 fraction bits, ties to even (8 = carry)
    code = (e << 3) + r;
    if (code > 0x7Eu) code = 0x7Eu;                      // saturate to 448
  } else {                                               // subnormal: |x| * 512 is exact
    float f;
    const uint32_t ab = a;
    memcpy(&f, &ab, 4);
#if defined(__HIP_DEVICE_COMPILE__)
    code = (uint32_t)__builtin_rintf(f * 512.0f);        // ties to even; 8 encodes 2^-6
#else
    code = (uint32_t)nearbyintf(f * 512.0f);             // default rounding mode: ties to even
#endif
  }
  return (uint8_t)(sign | code);
}

#if defined(__HIPCC__)
// The device encoder: the gfx950 conversion instruction (OCP E4M3, round to
// nearest even) on inputs clamped to +-448, two values per instruction.  For
// every fp32 input other than NaN it gives f32_to_e4m3's code
// (fdkv_check_conversions compares the two over all 2^32 bit patterns); the
// stored coefficients are finite.  Writes the
// codes of a and b to bytes 0-1 (hi = false) or 2-3 (hi = true) of old.
__device__ __forceinline__ uint32_t e4m3_pair(float a, float b, uint32_t old, bool hi) {
  const float ca = __builtin_amdgcn_fmed3f(a, -448.f, 448.f), cb = __builtin_amdgcn_fmed3f(b, -448.f, 448.f);
  return hi ? (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(ca, cb, (int)old, true)
            : (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(ca, cb, (int)old, false);
}
__device__ __forceinline__ uint32_t e4m3_quad(float a, float b, float c, float d) {
  return e4m3_pair(c, d, e4m3_pair(a, b, 0u, false), true);
}
__device__ __forceinline__ uint8_t e4m3_one(float a) { return (uint8_t)e4m3_pair(a, 0.f, 0u, false); }
#endif

}  // namespace fdkv
