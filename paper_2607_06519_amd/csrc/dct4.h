// High-frequency coefficients of the orthonormal DCT-II(4) along depth, as
// the blocks of four rank and store them (Section 3, Eq. 1 with B = 4).
//
// Z_j = sum_n F_4[j][n] x_n with F_4[j][n] = cos(pi (2n+1) j / 8) / sqrt(2);
// by the mirror symmetry of the basis this is the butterfly
//   Z_1 = a (x0 - x3) + b (x1 - x2)
//   Z_2 = ((x0 + x3) - (x1 + x2)) / 2
//   Z_3 = b (x0 - x3) - a (x1 - x2)
// with a = F_4[1][0], b = F_4[1][1].  Every product and sum is rounded on its
// own (no fused multiply-add), so the ranking is reproducible bit for bit.
// Plain C++, usable on the host.
#pragma once

#if defined(__HIPCC__)
#define FDKV_DCT4_HD __host__ __device__ __forceinline__
#else
#define FDKV_DCT4_HD inline
#endif

namespace fdkv {

// cos(pi/8)/sqrt(2) and cos(3pi/8)/sqrt(2), rounded to fp32
constexpr float kDct4A = 0x1.4e7aeap-1f;
constexpr float kDct4B = 0x1.1517a8p-2f;

FDKV_DCT4_HD void dct4_high(float x0, float x1, float x2, float x3, float& z1, float& z2, float& z3) {
#pragma clang fp contract(off)
  const float d03 = x0 - x3, d12 = x1 - x2;
  const float s03 = x0 + x3, s12 = x1 + x2;
  z1 = kDct4A * d03 + kDct4B * d12;
  z2 = (s03 - s12) * 0.5f;
  z3 = kDct4B * d03 - kDct4A * d12;
}

}  // namespace fdkv
