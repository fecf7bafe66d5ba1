// Per-token top-k channel selection for the sparse high-frequency residual.
//
// One lane owns one token.  Keys are the bit patterns of |fl32(x[2b] - x[2b+1])|
// (non-negative floats order like unsigned integers).  The k largest keys are
// kept, ties going to the lower channel, and the kept channels are produced in
// ascending order.
//
// Threshold: tau, the k-th largest key counted with multiplicity, comes from a
// comparator network in registers: groups of GS keys (GS = the power of two at
// or above k) are sorted by a bitonic network, then pairs of sorted groups are
// merged keeping only their top GS (elementwise max against the reversed
// partner gives a bitonic sequence holding the top GS, which a half-cleaner
// cascade sorts).  Selection: every key above tau, then the lowest channels
// whose key equals tau until k are chosen.
//
// Blocks of four rank 3D keys per token with a streaming variant
// (absorb16, list_threshold): see below.
//
// Everything here is plain C++ usable on the host, so the network can be
// checked on the CPU against a sort.
#pragma once
#include <stdint.h>

#if defined(__HIPCC__)
#define FDKV_NET_HD __host__ __device__ __forceinline__
#else
#define FDKV_NET_HD inline
#endif

namespace fdkv {
namespace net {

FDKV_NET_HD void ce_desc(uint32_t& x, uint32_t& y) {
  const uint32_t hi = x > y ? x : y;
  const uint32_t lo = x > y ? y : x;
  x = hi;
  y = lo;
}

// Sort a[0..N) descending (N a power of two).
template <int N>
FDKV_NET_HD void sort_desc(uint32_t* a) {
#pragma unroll
  for (int size = 2; size <= N; size <<= 1) {
#pragma unroll
    for (int j = size >> 1; j > 0; j >>= 1) {
#pragma unroll
      for (int i = 0; i < N; ++i) {
        const int l = i ^ j;
        if (l > i) {
          if ((i & size) == 0)
            ce_desc(a[i], a[l]);
          else
            ce_desc(a[l], a[i]);
        }
      }
    }
  }
}

// Sort a bitonic sequence a[0..N) descending.
template <int N>
FDKV_NET_HD void merge_bitonic_desc(uint32_t* a) {
#pragma unroll
  for (int j = N >> 1; j > 0; j >>= 1) {
#pragma unroll
    for (int i = 0; i < N; ++i)
      if ((i & j) == 0) ce_desc(a[i], a[i + j]);
  }
}

// k-th largest of a[0..D) with multiplicity, 1 <= k <= GS <= D.  Destroys a.
template <int D, int GS>
FDKV_NET_HD uint32_t kth_largest(uint32_t* a, int k) {
  static_assert((GS & (GS - 1)) == 0 && GS <= D && D % GS == 0, "group size");
#pragma unroll
  for (int g = 0; g < D / GS; ++g) sort_desc<GS>(a + g * GS);
#pragma unroll
  for (int st = 1; st < D / GS; st <<= 1) {
#pragma unroll
    for (int g = 0; g < D / GS; g += 2 * st) {
      uint32_t* A = a + g * GS;
      uint32_t* B = a + (g + st) * GS;
#pragma unroll
      for (int i = 0; i < GS; ++i) A[i] = A[i] > B[GS - 1 - i] ? A[i] : B[GS - 1 - i];
      merge_bitonic_desc<GS>(A);
    }
  }
  uint32_t tau = a[0];
#pragma unroll
  for (int i = 1; i < GS; ++i)
    if (i == k - 1) tau = a[i];
  return tau;
}

// k-th largest of key[0..D) with multiplicity, 1 <= k <= RS, leaving the keys
// as they are (the selection mask reads them again).  A list R of the RS
// largest keys seen so far, sorted descending, absorbs one sorted group of RS
// keys at a time: the elementwise max of R against the group reversed is
// bitonic and holds the RS largest of both, and the half-cleaner cascade
// sorts it again.  The first group becomes R as it is.
template <int D, int RS>
FDKV_NET_HD uint32_t kth_largest_keep(const uint32_t* key, int k) {
  static_assert((RS & (RS - 1)) == 0 && RS <= D && D % RS == 0, "list size");
  uint32_t R[RS];
#pragma unroll
  for (int i = 0; i < RS; ++i) R[i] = key[i];
  sort_desc<RS>(R);
#pragma unroll
  for (int g = 1; g < D / RS; ++g) {
    uint32_t x[RS];
#pragma unroll
    for (int i = 0; i < RS; ++i) x[i] = key[g * RS + i];
    sort_desc<RS>(x);
#pragma unroll
    for (int i = 0; i < RS; ++i) R[i] = R[i] > x[RS - 1 - i] ? R[i] : x[RS - 1 - i];
    merge_bitonic_desc<RS>(R);
  }
  uint32_t tau = R[0];
#pragma unroll
  for (int i = 1; i < RS; ++i)
    if (i == k - 1) tau = R[i];
  return tau;
}

// Streaming form (blocks of four, 3D keys per token): a list R of the RS
// largest keys seen so far, sorted descending and starting at zero, absorbs
// a group of 16 keys (destroyed).  The elementwise max of R's last 16
// entries against the sorted group reversed leaves R bitonic and holding the
// RS largest of both; the half-cleaner cascade sorts it again.
template <int RS>
FDKV_NET_HD void absorb16(uint32_t* R, uint32_t* g) {
  static_assert(RS >= 16 && (RS & (RS - 1)) == 0, "list size");
  sort_desc<16>(g);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const uint32_t o = g[15 - i];
    R[RS - 16 + i] = R[RS - 16 + i] > o ? R[RS - 16 + i] : o;
  }
  merge_bitonic_desc<RS>(R);
}

// tau = the k-th largest key (1 <= k <= RS) and the number of keys equal to
// tau that a selection of k takes (k minus the keys above tau, all of which
// are in the list).
template <int RS>
FDKV_NET_HD uint32_t list_threshold(const uint32_t* R, int k, int* need_eq) {
  uint32_t tau = R[0];
#pragma unroll
  for (int i = 1; i < RS; ++i)
    if (i == k - 1) tau = R[i];
  int n = k;
#pragma unroll
  for (int i = 0; i < RS; ++i) n -= R[i] > tau ? 1 : 0;
  *need_eq = n;
  return tau;
}

FDKV_NET_HD int popc(uint32_t x) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __builtin_popcount(x);
#else
  int n = 0;
  while (x) {
    x &= x - 1;
    ++n;
  }
  return n;
#endif
}

FDKV_NET_HD int ctz32(uint32_t x) {  // x != 0
#if defined(__HIP_DEVICE_COMPILE__)
  return __builtin_ctz(x);
#else
  int n = 0;
  while (!(x & 1u)) {
    x >>= 1;
    ++n;
  }
  return n;
#endif
}

// Channel mask (bit c%32 of word c/32) of the selection given tau: all keys
// above tau plus the lowest-index keys equal to tau, k bits in total.
template <int D>
FDKV_NET_HD void select_mask(const uint32_t* key, uint32_t tau, int k, uint32_t* mask) {
  constexpr int NW = D / 32;
  uint32_t eq[NW];
  int ngt = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    uint32_t g = 0, e = 0;
#pragma unroll
    for (int b = 0; b < 32; ++b) {
      const uint32_t x = key[w * 32 + b];
      g |= (x > tau ? 1u : 0u) << b;
      e |= (x == tau ? 1u : 0u) << b;
    }
    mask[w] = g;
    eq[w] = e;
    ngt += popc(g);
  }
  for (int need = k - ngt; need > 0; --need) {
    bool done = false;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      if (!done && eq[w]) {
        const uint32_t low = eq[w] & (0u - eq[w]);
        mask[w] |= low;
        eq[w] ^= low;
        done = true;
      }
    }
  }
}

// Lowest set channel of the mask, cleared from it (mask must be non-empty).
template <int D>
FDKV_NET_HD int pop_lowest(uint32_t* mask) {
  constexpr int NW = D / 32;
  int c = 0;
  bool found = false;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    if (!found && mask[w]) {
      c = w * 32 + ctz32(mask[w]);
      mask[w] &= mask[w] - 1;
      found = true;
    }
  }
  return c;
}

}  // namespace net
}  // namespace fdkv
