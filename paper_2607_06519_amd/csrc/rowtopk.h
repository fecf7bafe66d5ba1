// Wavefront top-k of a token row (Section 3, the sparse high-frequency
// residual of Eq. 3): the k channels of largest |fl32(x[l] - x[l+1])| of a
// row, ties to the lower channel, found by the lanes that hold the row.
//
// A row of d channels sits on LPR consecutive lanes (a DPP row or part of
// one; 32 lanes for fp32 rows of 128 channels).  A lane's CPL keys form H
// segments of S = CPL / H consecutive channels: key s S + c of lane j is
// channel s LPR S + j S + c (H = 1: lane j holds channels CPL j ..
// CPL j + CPL - 1; H = 2: a lane holds one run in each half of the row, so
// that loads of a segment over the row's lanes are contiguous).  Keys are
// the bit patterns of the non-negative
// fp32 magnitudes, which order like the values.  Every lane of a row keeps
// the same bounds lo < hi with clo = #(keys >= lo) >= k and chi = #(keys >=
// hi) < k, and bisects [lo, hi) on the bit patterns, counting keys >= mid
// over the row with a DPP sum (two steps per round, one ballot per round).
// A row stops once clo = k (the selection is every key >= lo), hi = lo + 1
// (lo is the k-th largest key itself, and it is tied), or at most three
// keys lie in [lo, hi).  In the last case the k - chi keys still needed are
// either one (lo becomes the largest key below hi) or all but one (lo
// becomes the smallest key at or above lo), and the selection is every key
// above lo plus the first k - #(keys > lo) keys equal to lo in channel
// order (segment by segment, lanes in order within a segment).  The first lo is the smallest lane maximum (at least LPR keys reach
// it, so it is valid for k <= LPR), for LPR < k <= 2 LPR the smallest lane's
// second-largest key, else 0; the first hi is the row maximum plus one; an
// open row's interval halves every step, so every row stops within 32 steps.
// Returns the lane's selection as a CPL-bit mask.
#pragma once

#include "fdkv_common.h"

namespace fdkv {

#ifdef __HIPCC__

template <int LPR>
__device__ __forceinline__ uint32_t row_sum_u32(uint32_t x) {
  static_assert(LPR == 8 || LPR == 16 || LPR == 32, "row width");
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, kDppQuadXor1, 0xF, 0xF, false);
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, kDppQuadXor2, 0xF, 0xF, false);
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, kDppRowHalfMirror, 0xF, 0xF, false);
  if constexpr (LPR >= 16) x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, kDppRowMirror, 0xF, 0xF, false);
  if constexpr (LPR == 32) x += (uint32_t)__shfl_xor((int)x, 16, 64);
  return x;
}

template <int LPR, bool MAX>
__device__ __forceinline__ uint32_t row_ext_u32(uint32_t x) {
  auto op = [](uint32_t a, uint32_t b) { return MAX ? (a > b ? a : b) : (a < b ? a : b); };
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, kDppQuadXor1, 0xF, 0xF, false));
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, kDppQuadXor2, 0xF, 0xF, false));
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, kDppRowHalfMirror, 0xF, 0xF, false));
  if constexpr (LPR >= 16) x = op(x, (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, kDppRowMirror, 0xF, 0xF, false));
  if constexpr (LPR == 32) x = op(x, (uint32_t)__shfl_xor((int)x, 16, 64));
  return x;
}

// Inclusive prefix sum over the row's lanes, in lane order (DPP row shifts
// inside each 16-lane DPP row; a row of 32 lanes adds the lower half's total
// through row_bcast:15; a row of 8 lanes masks the shifts at its boundary).
template <int LPR>
__device__ __forceinline__ uint32_t row_prefix_u32(uint32_t x) {
  static_assert(LPR == 8 || LPR == 16 || LPR == 32, "row width");
  const int lr = (int)(threadIdx.x & (LPR - 1));
  uint32_t y = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, false);  // row_shr:1
  x += (LPR != 8 || lr >= 1) ? y : 0u;
  y = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, false);           // row_shr:2
  x += (LPR != 8 || lr >= 2) ? y : 0u;
  y = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, false);           // row_shr:4
  x += (LPR != 8 || lr >= 4) ? y : 0u;
  if constexpr (LPR >= 16) x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, false);  // row_shr:8
  if constexpr (LPR == 32) x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xA, 0xF, false);  // row_bcast:15
  return x;
}

// Keys of this lane's CPL channels >= x, summed over the row.
template <int LPR, int CPL>
__device__ __forceinline__ uint32_t row_count_ge(const uint32_t (&key)[CPL], uint32_t x) {
  uint32_t c = 0;
#pragma unroll
  for (int i = 0; i < CPL; ++i) c += key[i] >= x ? 1u : 0u;
  return row_sum_u32<LPR>(c);
}

// The lane's selected keys (bit i: key i, the channel given above) of the k
// largest keys of its row, ties to the lower channel.  0 <= k <= d.
template <int LPR, int CPL, int H = 1>
__device__ __forceinline__ uint32_t row_topk_mask(const uint32_t (&key)[CPL], int k) {
  static_assert(H >= 1 && CPL % H == 0 && CPL < 32, "segments, and one mask bit per key");
  constexpr int S = CPL / H;
  constexpr uint32_t kAll = (1u << CPL) - 1u;
  if (k <= 0) return 0u;
  if (k >= LPR * CPL) return kAll;
  uint32_t lmax = key[0];
#pragma unroll
  for (int i = 1; i < CPL; ++i) lmax = key[i] > lmax ? key[i] : lmax;
  const uint32_t rmax = row_ext_u32<LPR, true>(lmax);
  uint32_t lo = 0u;
  if (k <= LPR) {
    lo = row_ext_u32<LPR, false>(lmax);
  } else if (CPL >= 2 && k <= 2 * LPR) {
    // every lane's second-largest key: at least 2 LPR keys reach the smallest
    uint32_t m1 = 0u, m2 = 0u;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const uint32_t x = key[i];
      m2 = max(m2, min(m1, x));
      m1 = max(m1, x);
    }
    lo = row_ext_u32<LPR, false>(m2);
  }
  uint32_t hi = rmax + 1u;
  uint32_t clo = row_count_ge<LPR, CPL>(key, lo), chi = 0;
  const uint32_t ku = (uint32_t)k;
  // A stopped row may take further steps: they keep both invariants and
  // only shrink [lo, hi), so no per-row guard is needed inside a round.
  for (int round = 0; round < 20; ++round) {
    if (__ballot(clo != ku && hi - lo > 1u && clo - chi > 3u) == 0) break;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const uint32_t mid = lo + ((hi - lo) >> 1);
      const uint32_t c = row_count_ge<LPR, CPL>(key, mid);
      const bool up = c >= ku;
      lo = up ? mid : lo;
      clo = up ? c : clo;
      hi = up ? hi : mid;
      chi = up ? chi : c;
    }
  }
  {
    // at most three keys in [lo, hi): one more key needed, or one too many
    const uint32_t need = ku - chi, ns = clo - chi;
    const bool take_max = ns > need && need == 1u;
    const bool drop_min = ns > need && need + 1u == ns && !take_max;
    if (__ballot(take_max || drop_min) != 0) {
      // one max reduction for both: the largest key below hi, or the
      // complement of the smallest key at or above lo (complements order
      // the other way round)
      uint32_t m = 0;
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
        const uint32_t x = take_max ? (key[i] < hi ? key[i] : 0u) : (key[i] >= lo ? ~key[i] : 0u);
        m = x > m ? x : m;
      }
      m = row_ext_u32<LPR, true>(m);
      if (take_max) lo = m;
      if (drop_min) lo = ~m;
      clo = row_count_ge<LPR, CPL>(key, lo);
    }
  }
  uint32_t sel = 0;
#pragma unroll
  for (int i = 0; i < CPL; ++i) sel |= key[i] >= lo ? 1u << i : 0u;
  const bool tied = clo != ku;  // lo is the k-th largest key, and it is tied
  if (__ballot(tied) != 0) {
    // keys above lo, then the first equal keys in channel order
    const uint32_t cgt = row_count_ge<LPR, CPL>(key, lo + 1u);
    uint32_t eq = 0;
#pragma unroll
    for (int i = 0; i < CPL; ++i) eq |= key[i] == lo ? 1u << i : 0u;
    // rank of the lane's first equal key of each segment: the equal keys of
    // the row's earlier segments, then those of the segment's lower lanes
    uint32_t start[H];
    uint32_t base = 0;
#pragma unroll
    for (int sg = 0; sg < H; ++sg) {
      const uint32_t n = (uint32_t)__builtin_popcount(eq & (((1u << S) - 1u) << (sg * S)));
      start[sg] = base + row_prefix_u32<LPR>(n) - n;
      if (sg + 1 < H) base += row_sum_u32<LPR>(n);
    }
    if (tied) {
      const uint32_t need = ku - cgt;
      uint32_t s2 = 0;
#pragma unroll
      for (int sg = 0; sg < H; ++sg) {
        uint32_t rank = start[sg];
#pragma unroll
        for (int c = 0; c < S; ++c) {
          const int i = sg * S + c;
          if (key[i] > lo) s2 |= 1u << i;
          if (key[i] == lo) {
            if (rank < need) s2 |= 1u << i;
            ++rank;
          }
        }
      }
      sel = s2;
    }
  }
  return sel;
}

#endif  // __HIPCC__

}  // namespace fdkv
