// Prefill-time compression of the KV cache (Section 3, Eq. 1 and Eq. 3).
//
// Two kernels:
//  * compress_dense - coalesced streaming pass over every (pair, KV head):
//    shared/residual heads write the pair mean M = (x[2b] + x[2b+1]) / 2
//    (the per-layer image of the low-frequency DCT coefficient) for K and V;
//    exact heads copy the four input rows.
//  * residual_select - one lane per token: the top-k channels of
//    |fl32(x[2b] - x[2b+1])| by a register comparator network (topk_net.h),
//    written as ascending uint8 indices plus D = (x[2b] - x[2b+1]) / 2 at those
//    channels.  Used for residual heads (K and V independently) and by the
//    probe (K indices only, into its workspace).
#include "fdkv_common.h"
#include "fdkv_kernels.h"
#include "fp8.h"
#include "topk_net.h"

namespace fdkv {

// 16 bytes of inputs -> 16 bytes of pair means, fp32 arithmetic.
template <bool BF16>
__device__ __forceinline__ uint4 pair_mean(uint4 a, uint4 b) {
  uint4 r;
  uint32_t* pr = reinterpret_cast<uint32_t*>(&r);
  const uint32_t* pa = reinterpret_cast<const uint32_t*>(&a);
  const uint32_t* pb = reinterpret_cast<const uint32_t*>(&b);
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    if constexpr (BF16) {
      const float lo = (bf16_lo(pa[w]) + bf16_lo(pb[w])) * 0.5f;
      const float hi = (bf16_hi(pa[w]) + bf16_hi(pb[w])) * 0.5f;
      pr[w] = pack_bf16x2(lo, hi);
    } else {
      pr[w] = as_u32((as_f32(pa[w]) + as_f32(pb[w])) * 0.5f);
    }
  }
  return r;
}

// 16 bytes of bf16 inputs (8 channels) -> 8 bytes of FP8 E4M3 pair means.
__device__ __forceinline__ uint2 pair_mean_e4m3(uint4 a, uint4 b) {
  const uint32_t* pa = reinterpret_cast<const uint32_t*>(&a);
  const uint32_t* pb = reinterpret_cast<const uint32_t*>(&b);
  uint32_t w[2] = {0u, 0u};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t lo = f32_to_e4m3((bf16_lo(pa[i]) + bf16_lo(pb[i])) * 0.5f);
    const uint32_t hi = f32_to_e4m3((bf16_hi(pa[i]) + bf16_hi(pb[i])) * 0.5f);
    w[i >> 1] |= (lo | (hi << 8)) << (16 * (i & 1));
  }
  return make_uint2(w[0], w[1]);
}

template <int D, bool BF16>
__global__ __launch_bounds__(256) void compress_dense_kernel(CompressParams P) {
  constexpr int E = BF16 ? 2 : 4;
  constexpr int NP = D * E / 16;        // 16-byte pieces per row
  constexpr int RPP = 256 / NP;         // rows per pass
  const int unit = blockIdx.y;          // pair * Hkv + head
  const int pair = unit / P.hkv, head = unit % P.hkv;
  const int mode = P.modes[unit];
  const int T = P.seq_len;
  const uint64_t row_bytes = (uint64_t)D * E;
  const uint64_t head_off = (uint64_t)head * T * row_bytes;
  const uint8_t* k0 = static_cast<const uint8_t*>(P.k[2 * pair]) + head_off;
  const uint8_t* k1 = static_cast<const uint8_t*>(P.k[2 * pair + 1]) + head_off;
  const uint8_t* v0 = static_cast<const uint8_t*>(P.v[2 * pair]) + head_off;
  const uint8_t* v1 = static_cast<const uint8_t*>(P.v[2 * pair + 1]) + head_off;
  uint8_t* seg = P.cache + P.seg_off[unit];
  const bool c8 = BF16 && P.coef8;      // shared planes in FP8 E4M3: 8 bytes per 16-byte input piece
  const SegLayout L = seg_layout(mode, T, D, P.topk, E, c8 ? 1 : E);
  const int piece = threadIdx.x % NP;
  const int row0 = blockIdx.x * kCompressTile + threadIdx.x / NP;
#pragma unroll 2
  for (int r = 0; r < kCompressTile; r += RPP) {
    const int t = row0 + r;
    if (t >= T) break;
    const uint64_t off = (uint64_t)t * row_bytes + piece * 16;
    const uint4 ka = *reinterpret_cast<const uint4*>(k0 + off);
    const uint4 kb = *reinterpret_cast<const uint4*>(k1 + off);
    const uint4 va = *reinterpret_cast<const uint4*>(v0 + off);
    const uint4 vb = *reinterpret_cast<const uint4*>(v1 + off);
    if (mode == kExact) {
      *reinterpret_cast<uint4*>(seg + L.k0 + off) = ka;
      *reinterpret_cast<uint4*>(seg + L.k1 + off) = kb;
      *reinterpret_cast<uint4*>(seg + L.v0 + off) = va;
      *reinterpret_cast<uint4*>(seg + L.v1 + off) = vb;
    } else if (c8) {
      const uint64_t o8 = (uint64_t)t * D + piece * 8;
      *reinterpret_cast<uint2*>(seg + L.mk + o8) = pair_mean_e4m3(ka, kb);
      *reinterpret_cast<uint2*>(seg + L.mv + o8) = pair_mean_e4m3(va, vb);
    } else {
      *reinterpret_cast<uint4*>(seg + L.mk + off) = pair_mean<BF16>(ka, kb);
      *reinterpret_cast<uint4*>(seg + L.mv + off) = pair_mean<BF16>(va, vb);
    }
  }
}

// ---------------------------------------------------------------- residual select
// LDS holds fp32 differences of 64 tokens, [token][D] in float4 units whose
// index is XOR-swizzled with the token so that one-row-per-lane reads are
// free of bank conflicts.
template <int D>
__device__ __forceinline__ int diff_slot(int t, int j) {  // float4 index
  return t * (D / 4) + (j ^ (t & 15));
}

template <int D, bool BF16, int GS>
__global__ __launch_bounds__(64) void residual_select_kernel(SelectParams P) {
  constexpr int E = BF16 ? 2 : 4;
  constexpr int NP = D * E / 16;
  constexpr int CPP = 16 / E;           // channels per input piece
  constexpr int RPI = 64 / NP;          // rows per load instruction
  constexpr int NW = D / 32;
  __shared__ float4 diff[64 * D / 4];

  const int unit = blockIdx.y;
  const int tensor = blockIdx.z;        // 0: K, 1: V
  if (P.modes && P.modes[unit] != kResidual) return;
  const int pair = unit / P.hkv, head = unit % P.hkv;
  const int T = P.seq_len, k = P.topk;
  const int lane = threadIdx.x;
  const int tok0 = blockIdx.x * 64;
  const uint64_t row_bytes = (uint64_t)D * E;
  const void* const* src = tensor ? P.v : P.k;
  const uint64_t head_off = (uint64_t)head * T * row_bytes;
  const uint8_t* xa = static_cast<const uint8_t*>(src[2 * pair]) + head_off;
  const uint8_t* xb = static_cast<const uint8_t*>(src[2 * pair + 1]) + head_off;

  // 1. coalesced load of 64 rows, differences into LDS
  {
    const int piece = lane % NP;
#pragma unroll 4
    for (int r = lane / NP; r < 64; r += RPI) {
      const int t = min(tok0 + r, T - 1);
      const uint64_t off = (uint64_t)t * row_bytes + piece * 16;
      const uint4 a = *reinterpret_cast<const uint4*>(xa + off);
      const uint4 b = *reinterpret_cast<const uint4*>(xb + off);
      const uint32_t* pa = reinterpret_cast<const uint32_t*>(&a);
      const uint32_t* pb = reinterpret_cast<const uint32_t*>(&b);
      float d[CPP];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        if constexpr (BF16) {
          d[2 * w] = bf16_lo(pa[w]) - bf16_lo(pb[w]);
          d[2 * w + 1] = bf16_hi(pa[w]) - bf16_hi(pb[w]);
        } else {
          d[w] = as_f32(pa[w]) - as_f32(pb[w]);
        }
      }
#pragma unroll
      for (int q = 0; q < CPP / 4; ++q) {
        const int j = piece * (CPP / 4) + q;  // float4 index within the row
        diff[diff_slot<D>(r, j)] = make_float4(d[4 * q], d[4 * q + 1], d[4 * q + 2], d[4 * q + 3]);
      }
    }
  }
  __syncthreads();

  // 2. one lane per token: threshold by the comparator network, then the mask
  const int t = tok0 + lane;
  uint32_t mask[NW];
  {
    uint32_t key[D];
#pragma unroll
    for (int j = 0; j < D / 4; ++j) {
      const float4 v = diff[diff_slot<D>(lane, j)];
      key[4 * j + 0] = as_u32(v.x) & 0x7FFFFFFFu;
      key[4 * j + 1] = as_u32(v.y) & 0x7FFFFFFFu;
      key[4 * j + 2] = as_u32(v.z) & 0x7FFFFFFFu;
      key[4 * j + 3] = as_u32(v.w) & 0x7FFFFFFFu;
    }
    const uint32_t tau = net::kth_largest<D, GS>(key, k);
#pragma unroll
    for (int j = 0; j < D / 4; ++j) {
      const float4 v = diff[diff_slot<D>(lane, j)];
      key[4 * j + 0] = as_u32(v.x) & 0x7FFFFFFFu;
      key[4 * j + 1] = as_u32(v.y) & 0x7FFFFFFFu;
      key[4 * j + 2] = as_u32(v.z) & 0x7FFFFFFFu;
      key[4 * j + 3] = as_u32(v.w) & 0x7FFFFFFFu;
    }
    net::select_mask<D>(key, tau, k, mask);
  }
  if (t >= T) return;

  // 3. ascending channels, half differences, packed stores
  uint8_t* out_idx;
  uint8_t* out_val;
  const bool c8 = BF16 && P.coef8;      // residual values in FP8 E4M3
  const int CE = c8 ? 1 : E;            // bytes per stored value
  if (P.modes) {
    uint8_t* seg = P.cache + P.seg_off[unit];
    const SegLayout L = seg_layout(kResidual, T, D, k, E, CE);
    out_idx = seg + (tensor ? L.iv : L.ik);
    out_val = seg + (tensor ? L.vv : L.vk);
  } else {
    out_idx = P.idx_out + (uint64_t)unit * plane_bytes((uint64_t)T * k);
    out_val = nullptr;
  }
  out_idx += (uint64_t)t * k;
  if (out_val) out_val += (uint64_t)t * k * CE;
  const float* drow = reinterpret_cast<const float*>(diff);
  if ((k & 3) == 0 && k <= GS) {
    uint32_t iw[GS / 4];
    uint32_t vw[GS * E / 4];
#pragma unroll
    for (int s = 0; s < GS; ++s) {
      if (s < k) {
        const int c = net::pop_lowest<D>(mask);
        const float dv = drow[diff_slot<D>(lane, c >> 2) * 4 + (c & 3)] * 0.5f;
        if (s % 4 == 0) iw[s / 4] = 0;
        iw[s / 4] |= (uint32_t)c << (8 * (s % 4));
        if constexpr (BF16) {
          if (c8) {
            if (s % 4 == 0) vw[s / 4] = 0;
            vw[s / 4] |= (uint32_t)f32_to_e4m3(dv) << (8 * (s % 4));
          } else {
            if (s % 2 == 0) vw[s / 2] = 0;
            vw[s / 2] |= f32_to_bf16_bits(dv) << (16 * (s % 2));
          }
        } else {
          vw[s] = as_u32(dv);
        }
      }
    }
    uint32_t* oi = reinterpret_cast<uint32_t*>(out_idx);
#pragma unroll
    for (int w = 0; w < GS / 4; ++w)
      if (4 * w < k) oi[w] = iw[w];
    if (out_val) {
      uint32_t* ov = reinterpret_cast<uint32_t*>(out_val);
#pragma unroll
      for (int w = 0; w < GS * E / 4; ++w)
        if (w < k * CE / 4) ov[w] = vw[w];
    }
  } else {
    for (int s = 0; s < k; ++s) {
      const int c = net::pop_lowest<D>(mask);
      out_idx[s] = (uint8_t)c;
      if (out_val) {
        const float dv = drow[diff_slot<D>(lane, c >> 2) * 4 + (c & 3)] * 0.5f;
        if (c8)
          out_val[s] = f32_to_e4m3(dv);
        else if constexpr (BF16)
          reinterpret_cast<uint16_t*>(out_val)[s] = (uint16_t)f32_to_bf16_bits(dv);
        else
          reinterpret_cast<float*>(out_val)[s] = dv;
      }
    }
  }
}

// ---------------------------------------------------------------- launchers
template <int D, bool BF16>
static hipError_t launch_compress_t(const CompressParams& P, hipStream_t s) {
  const dim3 grid((P.seq_len + kCompressTile - 1) / kCompressTile, P.n_pairs * P.hkv);
  hipLaunchKernelGGL((compress_dense_kernel<D, BF16>), grid, dim3(256), 0, s, P);
  return hipGetLastError();
}

hipError_t launch_compress_dense(const CompressParams& P, hipStream_t s) {
  if (P.d == 128) return P.bf16 ? launch_compress_t<128, true>(P, s) : launch_compress_t<128, false>(P, s);
  return P.bf16 ? launch_compress_t<64, true>(P, s) : launch_compress_t<64, false>(P, s);
}

template <int D, bool BF16, int GS>
static hipError_t launch_select_t(const SelectParams& P, int tensors, hipStream_t s) {
  const dim3 grid((P.seq_len + 63) / 64, P.n_pairs * P.hkv, tensors);
  hipLaunchKernelGGL((residual_select_kernel<D, BF16, GS>), grid, dim3(64), 0, s, P);
  return hipGetLastError();
}

template <int D, bool BF16>
static hipError_t launch_select_d(const SelectParams& P, int tensors, hipStream_t s) {
  if (P.topk <= 8) return launch_select_t<D, BF16, 8>(P, tensors, s);
  if (P.topk <= 16) return launch_select_t<D, BF16, 16>(P, tensors, s);
  return launch_select_t<D, BF16, D>(P, tensors, s);
}

hipError_t launch_residual_select(const SelectParams& P, int tensors, hipStream_t s) {
  if (P.topk <= 0) return hipSuccess;
  if (P.d == 128) return P.bf16 ? launch_select_d<128, true>(P, tensors, s) : launch_select_d<128, false>(P, tensors, s);
  return P.bf16 ? launch_select_d<64, true>(P, tensors, s) : launch_select_d<64, false>(P, tensors, s);
}

}  // namespace fdkv
