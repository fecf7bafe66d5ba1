// Shared definitions of the HIP path: element types, the segment layout of
// the compressed cache (Eq. 3 storage), and wavefront helpers for gfx950.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dct4.h"

#define FDKV_HD __host__ __device__ __forceinline__

namespace fdkv {

constexpr int kPlaneAlign = 256;
constexpr int kMaxLayers = 256;

enum : int { kShared = 0, kResidual = 1, kExact = 2 };

// A unit's mode byte: bits 0-1 hold the mode; with token-level sets whose
// fraction is routed per unit, bits 2-4 hold the index of the residual
// head's fraction among the cache's candidate fractions (0 otherwise).
constexpr int kMaxRates = 8;
FDKV_HD int mode_of(uint32_t byte) { return (int)(byte & 3u); }
FDKV_HD int rate_of(uint32_t byte) { return (int)((byte >> 2) & 7u); }
// The byte names a mode and, on a residual unit of a cache with n_rates
// routed fractions, one of them; every other byte is invalid.
FDKV_HD bool unit_byte_ok(uint32_t byte, int n_rates) {
  const uint32_t m = byte & 3u, r = byte >> 2;
  return m <= (uint32_t)kExact && (r == 0 || (m == (uint32_t)kResidual && r < (uint32_t)n_rates));
}

FDKV_HD float as_f32(uint32_t u) { return __builtin_bit_cast(float, u); }
FDKV_HD uint32_t as_u32(float f) { return __builtin_bit_cast(uint32_t, f); }

FDKV_HD uint64_t plane_bytes(uint64_t n) { return (n + kPlaneAlign - 1) / kPlaneAlign * kPlaneAlign; }

// FP8 coefficient planes (the shared planes of an FP8 cache, one byte per
// channel) are stored in 1 KB blocks of R = 1024 / d token rows, so that a
// decode lane reads both of its rows' 8-channel pieces with one 16-byte
// load: piece p (channels 8p .. 8p + 7) of row t sits at
//   1024 * (t / R) + 16 * ((t % (R/2)) * (d/8) + p) + 8 * ((t % R) / (R/2)),
// i.e. rows t and t + R/2 of a block share a 16-byte slot.  The plane is
// padded to whole blocks.
constexpr int kC8Block = 1024;
FDKV_HD uint64_t c8_piece_offset(uint64_t t, int p, int d) {
  const uint64_t R = (uint64_t)(kC8Block / d), half = R / 2;
  const uint64_t r = t % R;
  return (t / R) * kC8Block + 16 * ((r % half) * (uint64_t)(d / 8) + (uint64_t)p) + 8 * (r / half);
}
FDKV_HD uint64_t coef_plane_bytes(uint64_t T, int d, int c) {
  const uint64_t n = T * (uint64_t)d * (uint64_t)c;
  return c == 1 ? plane_bytes((n + kC8Block - 1) / kC8Block * kC8Block) : plane_bytes(n);
}

// Byte offsets of the planes of one (sequence, block, KV head) segment of a
// block of B = 2 or 4 layers.
// Shared:   MK, MV.  Residual: MK, MV, IK, VK, IV, VV.
// Exact:    K of the B layers, then V of the B layers.
// Residual indices are uint8 channels (B = 2) or uint16 codes 4c + j (B = 4).
struct SegLayout {
  uint64_t mk, mv, ik, vk, iv, vv;  // shared / residual planes
  uint64_t ek[4], ev[4];            // exact planes, by position in the block
  uint64_t total;
};

FDKV_HD int index_bytes(int B) { return B == 2 ? 1 : 2; }

// e: bytes per input / exact-plane element; c: bytes per stored coefficient
// (shared planes and residual values; c < e for FP8 coefficients).
FDKV_HD SegLayout seg_layout(int mode, uint64_t T, int d, int k, int e, int c, int B) {
  SegLayout s{};
  const uint64_t dense = plane_bytes(T * (uint64_t)d * e);
  const uint64_t coef = coef_plane_bytes(T, d, c);
  const uint64_t ip = plane_bytes(T * (uint64_t)k * index_bytes(B));
  const uint64_t vp = plane_bytes(T * (uint64_t)k * c);
  if (mode == kExact) {
    for (int i = 0; i < B; ++i) {
      s.ek[i] = i * dense;
      s.ev[i] = (B + i) * dense;
    }
    s.total = 2 * B * dense;
    return s;
  }
  s.mk = 0;
  s.mv = coef;
  s.total = 2 * coef;
  if (mode == kResidual) {
    s.ik = 2 * coef;
    s.vk = s.ik + ip;
    s.iv = s.vk + vp;
    s.vv = s.iv + ip;
    s.total = s.vv + vp;
  }
  return s;
}

// Token-level residual set (residual heads keep every high-frequency
// coefficient of n tokens): the shared planes, a 1-bit token mask
// (ceil(T/32) uint32 words), the count of residual tokens before every
// 128-token chunk (ceil(T/128) + 1 uint32), then the K and V rows of the n
// tokens, each (B - 1) x d coefficients.
constexpr int kTokChunk = 128;

struct TokLayout {
  uint64_t mk, mv, mask, count, hk, hv, total;
};

FDKV_HD uint64_t residual_token_count(uint64_t T, int ppm) { return (T * (uint64_t)ppm + 999999) / 1000000; }

FDKV_HD TokLayout tok_layout(int mode, uint64_t T, int d, int ppm, int e, int c, int B) {
  TokLayout s{};
  const uint64_t coef = coef_plane_bytes(T, d, c);
  if (mode == kExact) {
    s.total = 2 * B * plane_bytes(T * (uint64_t)d * e);
    return s;
  }
  s.mk = 0;
  s.mv = coef;
  s.total = 2 * coef;
  if (mode == kResidual) {
    const uint64_t n = residual_token_count(T, ppm);
    s.mask = 2 * coef;
    s.count = s.mask + plane_bytes((T + 31) / 32 * 4);
    s.hk = s.count + plane_bytes(((T + kTokChunk - 1) / kTokChunk + 1) * 4);
    s.hv = s.hk + plane_bytes(n * (uint64_t)(B - 1) * d * c);
    s.total = s.hv + plane_bytes(n * (uint64_t)(B - 1) * d * c);
  }
  return s;
}

// ---------------------------------------------------------------- bf16
FDKV_HD float bf16_lo(uint32_t w) { return as_f32(w << 16); }
FDKV_HD float bf16_hi(uint32_t w) { return as_f32(w & 0xFFFF0000u); }
FDKV_HD float bf16_to_f32(uint16_t h) { return as_f32((uint32_t)h << 16); }

#ifdef __HIPCC__
// Two fp32 values as a bf16 pair, round to nearest even: the gfx950
// conversion instruction, one per pair.  For every input other than NaN it
// gives the integer rounding below, subnormals and infinities included
// (fdkv_check_conversions compares the two over all 2^32 bit patterns).
__device__ __forceinline__ uint32_t cvt_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
  typedef float f32x2v __attribute__((ext_vector_type(2)));
  const f32x2v v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2v));
}
#endif

// Round to nearest even in integer arithmetic; inputs are not NaN.
FDKV_HD uint32_t bf16_bits_int(float f) {
  uint32_t u = as_u32(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}
// The same rounding: device code takes the conversion instruction, host
// code the integer form.
FDKV_HD uint32_t f32_to_bf16_bits(float f) {
#if defined(__HIP_DEVICE_COMPILE__)
  return cvt_bf16x2(f, 0.f) & 0xFFFFu;
#else
  return bf16_bits_int(f);
#endif
}
FDKV_HD uint32_t pack_bf16x2(float lo, float hi) {
#if defined(__HIP_DEVICE_COMPILE__)
  return cvt_bf16x2(lo, hi);
#else
  return f32_to_bf16_bits(lo) | (f32_to_bf16_bits(hi) << 16);
#endif
}

#ifdef __HIPCC__

// Two fp32 values as a sum of two bf16 pairs, hi = bf16(x) and
// lo = bf16(x - hi) (x - hi is exact in fp32): hi + lo is x to within
// 2^-18 |x|.  Products of bf16 values are exact in the fp32 MFMA, so the
// Gram matrix of x taken as H H^T + H L^T + L H^T carries only that error
// (plus the dropped L L^T, 2^-18 relative), where H H^T alone would carry
// the bf16 rounding of x (2^-9 relative per element).
__device__ __forceinline__ void split_bf16x2(float x0, float x1, uint32_t& hi, uint32_t& lo) {
  hi = cvt_bf16x2(x0, x1);
  lo = cvt_bf16x2(x0 - bf16_lo(hi), x1 - bf16_hi(hi));
}
#endif

// ---------------------------------------------------------------- wavefront helpers
// DPP lane permutations within rows of 16 lanes (gfx9 encodings).
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
constexpr int kDppQuadXor1 = 0xB1;     // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;     // quad_perm [2,3,0,1]
constexpr int kDppRowHalfMirror = 0x141;
constexpr int kDppRowMirror = 0x140;

// Sum over aligned groups of N lanes (N in 1,2,4,8,16); every lane gets its group's sum.
template <int N>
__device__ __forceinline__ float group_sum(float x) {
  if constexpr (N >= 2) x += dpp<kDppQuadXor1>(x);
  if constexpr (N >= 4) x += dpp<kDppQuadXor2>(x);
  if constexpr (N >= 8) x += dpp<kDppRowHalfMirror>(x);
  if constexpr (N >= 16) x += dpp<kDppRowMirror>(x);
  return x;
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

}  // namespace fdkv
