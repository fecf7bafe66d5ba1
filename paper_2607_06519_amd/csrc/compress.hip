// Prefill-time compression of the KV cache (Section 3, Eq. 1 and Eq. 3).
//
// Kernels:
//  * compress_dense - coalesced streaming pass over every (block, KV head):
//    shared/residual heads write the block mean M (the per-layer image of
//    the low-frequency DCT coefficient, the same for every layer of the
//    block) for K and V; exact heads copy the input rows.
//  * residual_select_reg (B = 2, k <= 16) and residual_select (B = 2, any
//    k) - one lane per token: the top-k channels of |fl32(x[2b] - x[2b+1])|
//    by a register comparator network (topk_net.h), written as ascending
//    uint8 indices plus D = (x[2b] - x[2b+1]) / 2 at those channels.
//  * residual_select4 (B = 4) - one lane per token: the top-k of the 3d
//    high-frequency coefficients Z_j[c] (j = 1..3) of the DCT-II(4), ranked
//    by |Z| as the fp32 butterfly gives them, written as ascending uint16
//    codes 4c + j plus Z_j[c].
// The select kernels serve residual heads (K and V independently) and the
// probe (K indices only, into its workspace).
#include "fdkv_common.h"
#include "fdkv_kernels.h"
#include "fp8.h"
#include "topk_net.h"

namespace fdkv {

// Channel i of a 16-byte piece, as fp32.
template <bool BF16>
__device__ __forceinline__ float chan(const uint4& v, int i) {
  const uint32_t* p = reinterpret_cast<const uint32_t*>(&v);
  if constexpr (BF16)
    return (i & 1) ? bf16_hi(p[i >> 1]) : bf16_lo(p[i >> 1]);
  else
    return as_f32(p[i]);
}

// Mean over the NB layers of channel i, fp32: (x0 + x1) / 2, or
// ((x0 + x3) + (x1 + x2)) / 4 (the butterfly order of the select kernel).
template <bool BF16, int NB>
__device__ __forceinline__ float block_mean(const uint4* x, int i) {
  if constexpr (NB == 2)
    return (chan<BF16>(x[0], i) + chan<BF16>(x[1], i)) * 0.5f;
  else
    return ((chan<BF16>(x[0], i) + chan<BF16>(x[3], i)) + (chan<BF16>(x[1], i) + chan<BF16>(x[2], i))) * 0.25f;
}

// 16 bytes of inputs per layer -> 16 bytes of block means in the input type.
template <bool BF16, int NB>
__device__ __forceinline__ uint4 mean_piece(const uint4* x) {
  uint4 r;
  uint32_t* pr = reinterpret_cast<uint32_t*>(&r);
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    if constexpr (BF16)
      pr[w] = pack_bf16x2(block_mean<true, NB>(x, 2 * w), block_mean<true, NB>(x, 2 * w + 1));
    else
      pr[w] = as_u32(block_mean<false, NB>(x, w));
  }
  return r;
}

// 16 bytes of bf16 inputs per layer (8 channels) -> 8 bytes of FP8 E4M3 block means.
template <int NB>
__device__ __forceinline__ uint2 mean_piece_e4m3(const uint4* x) {
  uint32_t w[2] = {0u, 0u};
#pragma unroll
  for (int i = 0; i < 8; ++i) w[i >> 2] |= (uint32_t)f32_to_e4m3(block_mean<true, NB>(x, i)) << (8 * (i & 3));
  return make_uint2(w[0], w[1]);
}

// The dense pass reads every input row once and writes every plane once:
// 16-byte loads and stores with the non-temporal cache hint.
typedef unsigned int u32x4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 load_stream(const uint8_t* p) {
  const u32x4v v = __builtin_nontemporal_load(reinterpret_cast<const u32x4v*>(p));
  return make_uint4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void store_stream(uint8_t* p, const uint4& x) {
  const u32x4v v = {x.x, x.y, x.z, x.w};
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4v*>(p));
}

template <int D, bool BF16, int NB>
__global__ __launch_bounds__(256) void compress_dense_kernel(CompressParams P) {
  constexpr int E = BF16 ? 2 : 4;
  constexpr int NP = D * E / 16;        // 16-byte pieces per row
  constexpr int RPP = 256 / NP;         // rows per pass
  const int bi = blockIdx.y / P.hkv, head = blockIdx.y % P.hkv;
  const int first = P.bl.first[bi];
  const int unit = P.bl.block[bi] * P.hkv + head;
  const int mode = mode_of(P.modes[unit]);
  const int T = P.seq_len;
  const uint64_t row_bytes = (uint64_t)D * E;
  const uint64_t head_off = (uint64_t)head * T * row_bytes;
  const uint8_t* kx[NB];
  const uint8_t* vx[NB];
#pragma unroll
  for (int n = 0; n < NB; ++n) {
    kx[n] = static_cast<const uint8_t*>(P.k[first + n]) + head_off;
    vx[n] = static_cast<const uint8_t*>(P.v[first + n]) + head_off;
  }
  uint8_t* seg = P.cache + P.seg_off[unit];
  const bool c8 = BF16 && P.coef8;      // shared planes in FP8 E4M3: 8 bytes per 16-byte input piece
  const SegLayout L = seg_layout(mode, T, D, P.topk, E, c8 ? 1 : E, NB);
  const int piece = threadIdx.x % NP;
  const int row0 = blockIdx.x * kCompressTile + threadIdx.x / NP;
#pragma unroll 2
  for (int r = 0; r < kCompressTile; r += RPP) {
    const int t = row0 + r;
    if (t >= T) break;
    const uint64_t off = (uint64_t)t * row_bytes + piece * 16;
    uint4 ka[NB], va[NB];
#pragma unroll
    for (int n = 0; n < NB; ++n) {
      ka[n] = load_stream(kx[n] + off);
      va[n] = load_stream(vx[n] + off);
    }
    if (mode == kExact) {
#pragma unroll
      for (int n = 0; n < NB; ++n) {
        store_stream(seg + L.ek[n] + off, ka[n]);
        store_stream(seg + L.ev[n] + off, va[n]);
      }
    } else if (c8) {
      const uint64_t o8 = (uint64_t)t * D + piece * 8;
      *reinterpret_cast<uint2*>(seg + L.mk + o8) = mean_piece_e4m3<NB>(ka);
      *reinterpret_cast<uint2*>(seg + L.mv + o8) = mean_piece_e4m3<NB>(va);
    } else {
      store_stream(seg + L.mk + off, mean_piece<BF16, NB>(ka));
      store_stream(seg + L.mv + off, mean_piece<BF16, NB>(va));
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

  const int bi = blockIdx.y / P.hkv, head = blockIdx.y % P.hkv;
  const int first = P.bl.first[bi];
  const int unit = P.bl.block[bi] * P.hkv + head;
  const int tensor = blockIdx.z;        // 0: K, 1: V
  if (P.modes && mode_of(P.modes[unit]) != kResidual) return;
  const int T = P.seq_len, k = P.topk;
  const int lane = threadIdx.x;
  const int tok0 = blockIdx.x * 64;
  const uint64_t row_bytes = (uint64_t)D * E;
  const void* const* src = tensor ? P.v : P.k;
  const uint64_t head_off = (uint64_t)head * T * row_bytes;
  const uint8_t* xa = static_cast<const uint8_t*>(src[first]) + head_off;
  const uint8_t* xb = static_cast<const uint8_t*>(src[first + 1]) + head_off;

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
    const SegLayout L = seg_layout(kResidual, T, D, k, E, CE, 2);
    out_idx = seg + (tensor ? L.iv : L.ik);
    out_val = seg + (tensor ? L.vv : L.vk);
  } else {
    out_idx = P.idx_out + (uint64_t)unit * probe_idx_stride(T, k);
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

// ---------------------------------------------------------------- residual select, k <= 16
// One lane per token with every key in registers: the lane loads its own
// rows of both layers (16-byte pieces), forms the fp32 differences, keeps
// their magnitudes as keys and, when a cache is written, puts the rounded
// half differences into an LDS table (16-byte pieces rotated by the lane).
// The threshold comes from the running sorted list of kth_largest_keep,
// which leaves the keys for the selection mask, so nothing goes through LDS
// on the way to the threshold and a workgroup needs only the value table:
// two waves fit on a SIMD instead of one.
template <int D, bool BF16>
__device__ __forceinline__ int vtab_slot(int lane, int piece) {  // 16-byte slot of a value piece
  constexpr int NPV = D * (BF16 ? 2 : 4) / 16;
  return lane * NPV + (piece ^ (lane & (NPV - 1)));
}

// C8: residual values stored as FP8 E4M3 (a compile-time flavour, so the
// bf16 path carries none of the encoder)
template <int D, bool BF16, int RS, bool C8>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(2))) void residual_select_reg_kernel(
    SelectParams P) {
  constexpr int E = BF16 ? 2 : 4;
  constexpr int NPC = D * E / 16;       // 16-byte pieces per input row
  constexpr int CPP = 16 / E;           // channels per piece
  constexpr int NW = D / 32;
  // value table: per lane D values of E bytes (bf16 bits, an E4M3 code in
  // the low byte, or fp32), piece p of the row holding channels p*CPP ...
  __shared__ uint4 vtab[64 * NPC];

  const int bi = blockIdx.y / P.hkv, head = blockIdx.y % P.hkv;
  const int first = P.bl.first[bi];
  const int unit = P.bl.block[bi] * P.hkv + head;
  const int tensor = blockIdx.z;        // 0: K, 1: V
  if (P.modes && mode_of(P.modes[unit]) != kResidual) return;
  const int T = P.seq_len, k = P.topk;
  const int lane = threadIdx.x;
  const int t = blockIdx.x * 64 + lane;
  const uint64_t row_bytes = (uint64_t)D * E;
  const void* const* src = tensor ? P.v : P.k;
  const uint64_t row = (uint64_t)head * T + (uint64_t)min(t, T - 1);
  const uint4* xa = reinterpret_cast<const uint4*>(static_cast<const uint8_t*>(src[first]) + row * row_bytes);
  const uint4* xb = reinterpret_cast<const uint4*>(static_cast<const uint8_t*>(src[first + 1]) + row * row_bytes);
  const bool values = P.modes != nullptr;
  constexpr bool c8 = BF16 && C8;

  uint32_t key[D];
#pragma unroll
  for (int p = 0; p < NPC; ++p) {
    const uint4 a = xa[p], b = xb[p];
    const uint32_t pa[4] = {a.x, a.y, a.z, a.w}, pb[4] = {b.x, b.y, b.z, b.w};
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
    for (int i = 0; i < CPP; ++i) key[p * CPP + i] = as_u32(d[i]) & 0x7FFFFFFFu;
    if (values) {
      uint32_t vw[4];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        if constexpr (BF16) {
          const float h0 = d[2 * w] * 0.5f, h1 = d[2 * w + 1] * 0.5f;
          if constexpr (c8)
            vw[w] = (uint32_t)f32_to_e4m3(h0) | ((uint32_t)f32_to_e4m3(h1) << 16);
          else
            vw[w] = cvt_bf16x2(h0, h1);
        } else {
          vw[w] = as_u32(d[w] * 0.5f);
        }
      }
      vtab[vtab_slot<D, BF16>(lane, p)] = make_uint4(vw[0], vw[1], vw[2], vw[3]);
    }
  }
  const uint32_t tau = net::kth_largest_keep<D, RS>(key, k);
  uint32_t mask[NW];
  net::select_mask<D>(key, tau, k, mask);
  if (t >= T) return;

  // ascending channels, packed stores
  constexpr int CE = c8 ? 1 : E;        // bytes per stored value
  uint8_t* out_idx;
  uint8_t* out_val = nullptr;
  if (values) {
    uint8_t* seg = P.cache + P.seg_off[unit];
    const SegLayout L = seg_layout(kResidual, T, D, k, E, CE, 2);
    out_idx = seg + (tensor ? L.iv : L.ik) + (uint64_t)t * k;
    out_val = seg + (tensor ? L.vv : L.vk) + (uint64_t)t * k * CE;
  } else {
    out_idx = P.idx_out + (uint64_t)unit * probe_idx_stride(T, k) + (uint64_t)t * k;
  }
  const uint8_t* vt = reinterpret_cast<const uint8_t*>(vtab);
  auto value_bits = [&](int c) -> uint32_t {  // stored value of channel c
    const uint8_t* pc = vt + vtab_slot<D, BF16>(lane, c / CPP) * 16 + (c % CPP) * E;
    if constexpr (BF16) return *reinterpret_cast<const uint16_t*>(pc) & (c8 ? 0xFFu : 0xFFFFu);
    else return *reinterpret_cast<const uint32_t*>(pc);
  };
  if ((k & 3) == 0) {
    uint32_t iw[RS / 4];
    uint32_t vw[RS * 4 / 4];
#pragma unroll
    for (int s = 0; s < RS; ++s) {
      if (s < k) {
        const int c = net::pop_lowest<D>(mask);
        if (s % 4 == 0) iw[s / 4] = 0;
        iw[s / 4] |= (uint32_t)c << (8 * (s % 4));
        if (values) {
          const uint32_t v = value_bits(c);
          if (CE == 1) {
            if (s % 4 == 0) vw[s / 4] = 0;
            vw[s / 4] |= v << (8 * (s % 4));
          } else if (CE == 2) {
            if (s % 2 == 0) vw[s / 2] = 0;
            vw[s / 2] |= v << (16 * (s % 2));
          } else {
            vw[s] = v;
          }
        }
      }
    }
    uint32_t* oi = reinterpret_cast<uint32_t*>(out_idx);
#pragma unroll
    for (int w = 0; w < RS / 4; ++w)
      if (4 * w < k) oi[w] = iw[w];
    if (values) {
      uint32_t* ov = reinterpret_cast<uint32_t*>(out_val);
#pragma unroll
      for (int w = 0; w < RS; ++w)
        if (w < k * CE / 4) ov[w] = vw[w];
    }
  } else {
    for (int s = 0; s < k; ++s) {
      const int c = net::pop_lowest<D>(mask);
      out_idx[s] = (uint8_t)c;
      if (values) {
        const uint32_t v = value_bits(c);
        if (CE == 1)
          out_val[s] = (uint8_t)v;
        else if (CE == 2)
          reinterpret_cast<uint16_t*>(out_val)[s] = (uint16_t)v;
        else
          reinterpret_cast<uint32_t*>(out_val)[s] = v;
      }
    }
  }
}

// ---------------------------------------------------------------- residual select, blocks of four
// The coefficients of the token's block come 16 channels at a time: the
// wave loads those channels of its 64 tokens from the four layers
// (coalesced), evaluates the DCT-II(4) butterfly in fp32 with every product
// and sum rounded on its own, and leaves Z_1..Z_3 in LDS, [token][channel][j]
// (float4 slots rotated by the token so one-row-per-lane reads spread over
// the banks).  Each lane then reads its token's 48 values.
//  pass 1 - threshold: a running list of the RS largest keys (sorted
//           descending) absorbs each sorted group of 16 keys (one frequency
//           of one chunk) by the bitonic merge of topk_net.h; tau is its
//           k-th entry and the list holds every key above tau.
//  pass 2 - selection in code order (channel, then frequency): every key
//           above tau and the first keys equal to tau until k are taken;
//           each candidate is written to the lane's LDS slot at its running
//           count, which advances only when it is taken (the count stops at
//           k, hence k + 1 slots), and the k slots are then stored as packed
//           words.
__device__ __forceinline__ int z4_slot(int t, int q) {  // float4 slot of quarter q (0..11) of token t's row
  return t * 12 + (q + t) % 12;
}

template <int D, bool BF16, int RS>
__global__ __launch_bounds__(64) void residual_select4_kernel(SelectParams P) {
  constexpr int E = BF16 ? 2 : 4;
  constexpr int CPP = 16 / E;           // channels per input piece
  constexpr int PPC = 16 / CPP;         // pieces per chunk of 16 channels
  constexpr int NC = D / 16;            // chunks
  __shared__ float4 zs[64 * 12];        // [token][16 channels][3] of one chunk
  __shared__ uint2 slot[64 * (RS + 1)];  // per lane: (code, value bits) of the taken entries

  const int bi = blockIdx.y / P.hkv, head = blockIdx.y % P.hkv;
  const int first = P.bl.first[bi];
  const int unit = P.bl.block[bi] * P.hkv + head;
  const int tensor = blockIdx.z;        // 0: K, 1: V
  if (P.modes && mode_of(P.modes[unit]) != kResidual) return;
  const int T = P.seq_len, k = P.topk;
  const int lane = threadIdx.x;
  const int tok0 = blockIdx.x * 64;
  const uint64_t row_bytes = (uint64_t)D * E;
  const void* const* src = tensor ? P.v : P.k;
  const uint64_t head_off = (uint64_t)head * T * row_bytes;
  const uint8_t* x[4];
#pragma unroll
  for (int n = 0; n < 4; ++n) x[n] = static_cast<const uint8_t*>(src[first + n]) + head_off;

  // The workgroup is one wave, so the staging needs only wave-scope ordering
  // (LDS operations of a wave complete in order): no workgroup barrier, which
  // would also wait for the next chunk's loads already in flight.
  auto wave_sync = [] {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
  };
  uint4 vin[PPC][4];  // the next chunk's input pieces, loaded ahead of its use
  auto load = [&](int ch) {
#pragma unroll
    for (int i = 0; i < PPC; ++i) {
      const int r = lane / PPC + (64 / PPC) * i, pc = lane % PPC;
      const int t = min(tok0 + r, T - 1);
      const uint64_t off = (uint64_t)t * row_bytes + (uint64_t)(ch * PPC + pc) * 16;
#pragma unroll
      for (int n = 0; n < 4; ++n) vin[i][n] = *reinterpret_cast<const uint4*>(x[n] + off);
    }
  };
  auto stage = [&]() {  // Z of the loaded chunk's 16 channels into LDS
    wave_sync();        // the previous chunk's rows are read
#pragma unroll
    for (int i = 0; i < PPC; ++i) {
      const int r = lane / PPC + (64 / PPC) * i, pc = lane % PPC;
      float z[3 * CPP];
#pragma unroll
      for (int c = 0; c < CPP; ++c)
        dct4_high(chan<BF16>(vin[i][0], c), chan<BF16>(vin[i][1], c), chan<BF16>(vin[i][2], c),
                  chan<BF16>(vin[i][3], c), z[3 * c], z[3 * c + 1], z[3 * c + 2]);
#pragma unroll
      for (int q = 0; q < 3 * CPP / 4; ++q)
        zs[z4_slot(r, pc * (3 * CPP / 4) + q)] = make_float4(z[4 * q], z[4 * q + 1], z[4 * q + 2], z[4 * q + 3]);
    }
    wave_sync();
  };
  auto row = [&](float (&zr)[48]) {
#pragma unroll
    for (int q = 0; q < 12; ++q) {
      const float4 v = zs[z4_slot(lane, q)];
      zr[4 * q] = v.x;
      zr[4 * q + 1] = v.y;
      zr[4 * q + 2] = v.z;
      zr[4 * q + 3] = v.w;
    }
  };

  // pass 1: the RS largest keys
  uint32_t R[RS];
#pragma unroll
  for (int i = 0; i < RS; ++i) R[i] = 0u;
  load(0);
  for (int ch = 0; ch < NC; ++ch) {
    stage();
    load(ch + 1 < NC ? ch + 1 : 0);  // the last one starts pass 2
    float zr[48];
    row(zr);
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      uint32_t g[16];
#pragma unroll
      for (int c = 0; c < 16; ++c) g[c] = as_u32(zr[3 * c + j]) & 0x7FFFFFFFu;
      net::absorb16<RS>(R, g);
    }
  }
  int need_eq;
  const uint32_t tau = net::list_threshold<RS>(R, k, &need_eq);

  // pass 2: selection in code order into the lane's slots
  uint2* my = slot + lane * (RS + 1);
  int s = 0, eq = 0;
  for (int ch = 0; ch < NC; ++ch) {
    stage();
    if (ch + 1 < NC) load(ch + 1);
    float zr[48];
    row(zr);
#pragma unroll
    for (int c = 0; c < 16; ++c)
#pragma unroll
      for (int j = 0; j < 3; ++j) {
        const float z = zr[3 * c + j];
        const uint32_t key = as_u32(z) & 0x7FFFFFFFu;
        const bool take = key > tau || (key == tau && eq < need_eq);
        eq += key == tau ? 1 : 0;
        my[s] = make_uint2((uint32_t)(4 * (16 * ch + c) + j + 1), as_u32(z));
        s += take ? 1 : 0;
      }
  }

  // store: codes as uint16, values in the coefficient type, packed in words
  const int t = tok0 + lane;
  if (t >= T) return;
  const bool c8 = BF16 && P.coef8;      // values in FP8 E4M3
  const int CE = c8 ? 1 : E;
  uint8_t* out_idx;
  uint8_t* out_val = nullptr;
  if (P.modes) {
    uint8_t* seg = P.cache + P.seg_off[unit];
    const SegLayout L = seg_layout(kResidual, T, D, k, E, CE, 4);
    out_idx = seg + (tensor ? L.iv : L.ik);
    out_val = seg + (tensor ? L.vv : L.vk);
  } else {
    out_idx = P.idx_out + (uint64_t)unit * probe_idx_stride(T, k);
  }
  auto value_bits = [&](int e) -> uint32_t {  // entry e in the coefficient type
    const float z = as_f32(my[e].y);
    if (c8) return f32_to_e4m3(z);
    if constexpr (BF16)
      return f32_to_bf16_bits(z);
    else
      return as_u32(z);
  };
  uint32_t* oi = reinterpret_cast<uint32_t*>(out_idx + (uint64_t)t * k * 2);
  if ((k & 1) == 0) {
#pragma unroll
    for (int w = 0; w < RS / 2; ++w)
      if (2 * w < k) oi[w] = my[2 * w].x | (my[2 * w + 1].x << 16);
  } else {
    for (int e = 0; e < k; ++e) reinterpret_cast<uint16_t*>(oi)[e] = (uint16_t)my[e].x;
  }
  if (!out_val) return;
  uint8_t* ov = out_val + (uint64_t)t * k * CE;
  if (CE == 4) {
#pragma unroll
    for (int e = 0; e < RS; ++e)
      if (e < k) reinterpret_cast<uint32_t*>(ov)[e] = value_bits(e);
  } else if (CE == 2 && (k & 1) == 0) {
#pragma unroll
    for (int w = 0; w < RS / 2; ++w)
      if (2 * w < k) reinterpret_cast<uint32_t*>(ov)[w] = value_bits(2 * w) | (value_bits(2 * w + 1) << 16);
  } else if (CE == 1 && (k & 3) == 0) {
#pragma unroll
    for (int w = 0; w < RS / 4; ++w)
      if (4 * w < k)
        reinterpret_cast<uint32_t*>(ov)[w] = value_bits(4 * w) | (value_bits(4 * w + 1) << 8) |
                                             (value_bits(4 * w + 2) << 16) | (value_bits(4 * w + 3) << 24);
  } else {
    for (int e = 0; e < k; ++e) {
      const uint32_t v = value_bits(e);
      if (CE == 1)
        ov[e] = (uint8_t)v;
      else
        reinterpret_cast<uint16_t*>(ov)[e] = (uint16_t)v;
    }
  }
}

// ---------------------------------------------------------------- launchers
template <int D, bool BF16, int NB>
static hipError_t launch_compress_t(const CompressParams& P, hipStream_t s) {
  const dim3 grid((P.seq_len + kCompressTile - 1) / kCompressTile, P.bl.n * P.hkv);
  hipLaunchKernelGGL((compress_dense_kernel<D, BF16, NB>), grid, dim3(256), 0, s, P);
  return hipGetLastError();
}

template <int NB>
static hipError_t launch_compress_b(const CompressParams& P, hipStream_t s) {
  if (P.d == 128) return P.bf16 ? launch_compress_t<128, true, NB>(P, s) : launch_compress_t<128, false, NB>(P, s);
  return P.bf16 ? launch_compress_t<64, true, NB>(P, s) : launch_compress_t<64, false, NB>(P, s);
}

hipError_t launch_compress_dense(const CompressParams& P, hipStream_t s) {
  if (P.bl.n == 0 || P.seq_len == 0) return hipSuccess;
  return P.bsize == 4 ? launch_compress_b<4>(P, s) : launch_compress_b<2>(P, s);
}

template <int D, bool BF16, int GS>
static hipError_t launch_select_t(const SelectParams& P, int tensors, hipStream_t s) {
  const dim3 grid((P.seq_len + 63) / 64, P.bl.n * P.hkv, tensors);
  hipLaunchKernelGGL((residual_select_kernel<D, BF16, GS>), grid, dim3(64), 0, s, P);
  return hipGetLastError();
}

template <int D, bool BF16, int RS>
static hipError_t launch_select_reg_t(const SelectParams& P, int tensors, hipStream_t s) {
  const dim3 grid((P.seq_len + 63) / 64, P.bl.n * P.hkv, tensors);
  if (BF16 && P.coef8)
    hipLaunchKernelGGL((residual_select_reg_kernel<D, BF16, RS, true>), grid, dim3(64), 0, s, P);
  else
    hipLaunchKernelGGL((residual_select_reg_kernel<D, BF16, RS, false>), grid, dim3(64), 0, s, P);
  return hipGetLastError();
}

template <int D, bool BF16>
static hipError_t launch_select_d(const SelectParams& P, int tensors, hipStream_t s) {
  if (P.topk <= 8) return launch_select_reg_t<D, BF16, 8>(P, tensors, s);
  if (P.topk <= 16) return launch_select_reg_t<D, BF16, 16>(P, tensors, s);
  return launch_select_t<D, BF16, D>(P, tensors, s);
}

template <int D, bool BF16, int RS>
static hipError_t launch_select4_t(const SelectParams& P, int tensors, hipStream_t s) {
  const dim3 grid((P.seq_len + 63) / 64, P.bl.n * P.hkv, tensors);
  hipLaunchKernelGGL((residual_select4_kernel<D, BF16, RS>), grid, dim3(64), 0, s, P);
  return hipGetLastError();
}

template <int D, bool BF16>
static hipError_t launch_select4_d(const SelectParams& P, int tensors, hipStream_t s) {
  if (P.topk <= 16) return launch_select4_t<D, BF16, 16>(P, tensors, s);
  if (P.topk <= 32) return launch_select4_t<D, BF16, 32>(P, tensors, s);
  if (P.topk <= 64) return launch_select4_t<D, BF16, 64>(P, tensors, s);
  return launch_select4_t<D, BF16, 128>(P, tensors, s);
}

hipError_t launch_residual_select(const SelectParams& P, int tensors, hipStream_t s) {
  if (P.topk <= 0 || P.bl.n == 0 || P.seq_len == 0) return hipSuccess;
  if (P.bsize == 4) {
    if (P.d == 128) return P.bf16 ? launch_select4_d<128, true>(P, tensors, s) : launch_select4_d<128, false>(P, tensors, s);
    return P.bf16 ? launch_select4_d<64, true>(P, tensors, s) : launch_select4_d<64, false>(P, tensors, s);
  }
  if (P.d == 128) return P.bf16 ? launch_select_d<128, true>(P, tensors, s) : launch_select_d<128, false>(P, tensors, s);
  return P.bf16 ? launch_select_d<64, true>(P, tensors, s) : launch_select_d<64, false>(P, tensors, s);
}

}  // namespace fdkv
