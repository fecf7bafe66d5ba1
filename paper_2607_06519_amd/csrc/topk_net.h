// Per-token top-k selection for the sparse high-frequency residual of blocks
// of four layers (Section 3, Eq. 3 with the DCT-II(4) of Eq. 1).
//
// One lane owns one token and ranks its 3D keys, the bit patterns of
// |Z_j[c]| (non-negative floats order like unsigned integers), in code order
// (channel, then frequency).  A list R of the RS largest keys seen so far,
// sorted descending, absorbs the keys 16 at a time (absorb16), and tau, the
// k-th largest key counted with multiplicity, is read from the list
// (list_threshold); the selection then takes every key above tau and the
// first keys equal to tau in code order until k are chosen.
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

}  // namespace net
}  // namespace fdkv
