// Online routing probe: the logit-reconstruction loss of Eq. (2).
//
// Pairs.  For a (pair b, KV head h) unit, let Delta_t be K^(m)_t - K_t of one
// layer of the pair.  With B = 2 the shared reconstruction misses -D_t for layer
// 2b and +D_t for layer 2b+1 (D = half the layer difference); the residual
// reconstruction misses the same vectors with the token's top-k channels
// zeroed (Dbar).  The squared logit errors summed over probe rows and tokens
// are therefore, for either layer,
//   sum_p sum_t (q_p . Delta_t)^2 = < C, S >,  C = sum_t Delta_t Delta_t^T,
//                                            S = sum_p q_p q_p^T,
// and the loss averaged over the pair's two layers and the G query heads is
//   E_m = < C_m, S_u > / (2 G P d),  S_u = sum over both layers' probe rows.
// Contracting the d x d Gram matrices instead of forming the (2 G P) x T
// logit matrices cuts the work from 2*(2GP)*T*d to 2*T*d^2 multiply-adds per
// mode (16x less at G = 4, P = 256, d = 128).
//
// Blocks of four.  Layer p of the block misses Delta_{p,t} = M_t - x_{p,t}
// (shared) or that plus the images F_4[j][p] Z_j[c] of the token's kept
// coefficients (residual); the layers now differ, so
//   E_m = sum_p < C_{p,m}, S_p > / (4 G P d)
// with one Gram matrix per layer of the deviations and of the probe rows.
//
// Kernels: probe_qgram forms the probe Gram matrices (MFMA
// Gram of the probe rows for bf16 queries, fp32 VALU for fp32 ones) into
// per-(layer, KV head) slots: a pair's S_u sits in the slot of its first
// layer, a block of four has one slot per layer; probe_dgram (pairs) and
// probe_dgram4 (blocks of four) stream the keys once, find each token's
// top-k in the same pass (the wavefront top-k of rowtopk.h, as compress
// does), and stage the bf16 deviations row-major in LDS; all Gram kernels
// take their
// v_mfma_f32_32x32x16_bf16 operands with transposing LDS reads
// (ds_read_b64_tr_b16) and accumulate the upper-triangular 32x32 blocks.
// The deviation Gram kernels contract with the probe Gram matrices in their
// epilogue and probe_finalize sums the per-workgroup partials in a fixed
// order in fp64.
#include "fdkv_common.h"
#include "fdkv_kernels.h"
#include "rowtopk.h"

namespace fdkv {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef short i16x8_t __attribute__((ext_vector_type(8)));
typedef i16x4_t __attribute__((address_space(3))) lds_i16x4_t;

namespace {

constexpr int kRsrcWord3 = 0x00020000;  // raw buffer, 32-bit data format (gfx9 family)
constexpr uint32_t kOobOff = 0x80000000u;  // past every input plane: buffer loads read 0
constexpr int kGramRows = 64;             // rows staged in LDS per step of the Gram kernels

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint64_t bytes) {
  const uint32_t n = bytes > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, kRsrcWord3);
}

__device__ __forceinline__ uint4 load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// Upper-triangular 32x32 blocks (I <= J) of a D x D Gram matrix, in order.
template <int NB>
struct TriTiles {
  int i[NB * (NB + 1) / 2], j[NB * (NB + 1) / 2];
  constexpr TriTiles() : i(), j() {
    int t = 0;
    for (int a = 0; a < NB; ++a)
      for (int b = a; b < NB; ++b) {
        i[t] = a;
        j[t] = b;
        ++t;
      }
  }
};

// Operand of v_mfma_f32_32x32x16_bf16 for channel block I and rows
// 16kk .. 16kk+15 of a row-major bf16 tile with LDR elements per row: lane l
// gets channel 32I + l%32 of rows 16kk + 8(l/32) .. +7, from two transposing
// reads.  In each 16-lane group, lane i of ds_read_b64_tr_b16 returns element
// i%4 of the 4-element row addressed by lane 4j + i/4 as its element j; the
// lanes therefore address rows base + i/4 at channels 32I + 16g + 4(i%4).
template <int LDR>
__device__ __forceinline__ bf16x8_t gram_operand(const uint16_t* tile, int kk, int I, int lane) {
  const int h = lane >> 5, g = (lane >> 4) & 1, li = lane & 15;
  const int row = 16 * kk + 8 * h + (li >> 2);
  const int col = 32 * I + 16 * g + 4 * (li & 3);
  const i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)(tile + row * LDR + col));
  const i16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)(tile + (row + 4) * LDR + col));
  const i16x8_t v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8_t, v);
}

// 32-bit word w of a 16-byte value.
__device__ __forceinline__ uint32_t word16(const uint4& v, int w) {
  return w == 0 ? v.x : w == 1 ? v.y : w == 2 ? v.z : v.w;
}

// Channel i of a 16-byte piece, as fp32.
template <bool BF16>
__device__ __forceinline__ float chan_of(const uint4& v, int i) {
  const uint32_t w = word16(v, BF16 ? i >> 1 : i);
  if constexpr (BF16)
    return (i & 1) ? bf16_hi(w) : bf16_lo(w);
  else
    return as_f32(w);
}

}  // namespace

template <int D, bool BF16>
__device__ __forceinline__ float load_q(const void* base, uint64_t i) {
  if constexpr (BF16)
    return bf16_to_f32(static_cast<const uint16_t*>(base)[i]);
  else
    return static_cast<const float*>(base)[i];
}

// One Gram slot of a launch: (list block bi, KV head, layer slot) from the
// workgroup index.  Pairs: one slot per unit summing the rows of both
// layers, stored at the pair's first layer.  Blocks of four: one slot per
// layer.
struct GramSlot {
  int layer, nl, head;
};
__device__ __forceinline__ GramSlot gram_slot(const ProbeParams& P, int x) {
  const int ns = P.bsize == 2 ? 1 : 4;
  const int bi = x / (P.hkv * ns), rem = x % (P.hkv * ns);
  GramSlot g;
  g.head = rem / ns;
  g.layer = P.bl.first[bi] + rem % ns;
  g.nl = P.bsize == 2 ? 2 : 1;
  return g;
}
__device__ __forceinline__ float* gram_at(const ProbeParams& P, int layer, int head) {
  return P.gram_q + ((uint64_t)layer * P.hkv + head) * P.d * P.d;
}

// S = sum of q q^T over the probe rows of the slot's layers and the G query heads.
template <int D, bool BF16>
__global__ __launch_bounds__(256) void probe_qgram_kernel(ProbeParams P) {
  constexpr int BS = D / 16;  // each thread owns a BS x BS block of S
  constexpr int RT = 32;      // rows per LDS tile
  __shared__ float rows[RT][D];
  const GramSlot gs = gram_slot(P, blockIdx.x);
  const int head = gs.head;
  const int G = P.hq / P.hkv, NP = P.n_probe;
  const int NR = gs.nl * G * NP;
  const int tid = threadIdx.x;
  const int bi = (tid / 16) * BS, bj = (tid % 16) * BS;
  float acc[BS][BS];
#pragma unroll
  for (int i = 0; i < BS; ++i)
#pragma unroll
    for (int j = 0; j < BS; ++j) acc[i][j] = 0.f;
  for (int r0 = 0; r0 < NR; r0 += RT) {
    __syncthreads();
    for (int i = tid; i < RT * D; i += 256) {
      const int rr = i / D, c = i % D, r = r0 + rr;
      float v = 0.f;
      if (r < NR) {
        const int ls = r / (G * NP), g = (r / NP) % G, p = r % NP;
        v = load_q<D, BF16>(P.qp[gs.layer + ls], ((uint64_t)(head * G + g) * NP + p) * D + c);
      }
      rows[rr][c] = v;
    }
    __syncthreads();
#pragma unroll 4
    for (int rr = 0; rr < RT; ++rr) {
      float a[BS], b[BS];
#pragma unroll
      for (int i = 0; i < BS; ++i) {
        a[i] = rows[rr][bi + i];
        b[i] = rows[rr][bj + i];
      }
#pragma unroll
      for (int i = 0; i < BS; ++i)
#pragma unroll
        for (int j = 0; j < BS; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
  }
  float* S = gram_at(P, gs.layer, head);
#pragma unroll
  for (int i = 0; i < BS; ++i)
#pragma unroll
    for (int j = 0; j < BS; ++j) S[(bi + i) * D + bj + j] = acc[i][j];
}

// S as the MFMA Gram matrix of the slot's bf16 probe rows (exact products,
// fp32 sums), upper-triangular 32x32 blocks only (the only ones the
// deviation kernels read).  One workgroup per slot; 64 rows per step, the
// next step's loads in flight during the current step's MFMAs; the four
// waves split the blocks.
template <int D>
__global__ __launch_bounds__(256) void probe_qgram_mfma_kernel(ProbeParams P) {
  constexpr int NPc = D / 8;                     // 16-byte pieces per row
  constexpr int NB = D / 32, NT = NB * (NB + 1) / 2;
  constexpr int TPW = (NT + 3) / 4;              // blocks per wave
  constexpr int R = kGramRows, LDR = D + 16;     // rows per step, LDS row stride (elements)
  constexpr int LPT = R * NPc / 256;             // loads per thread per step
  constexpr TriTiles<NB> tri{};
  __shared__ __attribute__((aligned(16))) uint16_t tile[R * LDR];
  const GramSlot gs = gram_slot(P, blockIdx.x);
  const int head = gs.head;
  const int G = P.hq / P.hkv, NP = P.n_probe;
  const int NR = gs.nl * G * NP;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const uint32_t RB = D * 2;
  const uint64_t span = (uint64_t)G * NP * RB;   // bytes of one layer's probe rows for this head
  const auto q0 = make_rsrc(static_cast<const uint8_t*>(P.qp[gs.layer]) + (uint64_t)head * span, span);
  const auto q1 = make_rsrc(static_cast<const uint8_t*>(P.qp[gs.layer + gs.nl - 1]) + (uint64_t)head * span, span);
  f32x16_t acc[TPW];
#pragma unroll
  for (int i = 0; i < TPW; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
  uint4 buf[LPT];
  auto load = [&](int r0) {
#pragma unroll
    for (int j = 0; j < LPT; ++j) {
      const int i = tid + 256 * j, r = r0 + i / NPc, pc = i % NPc;
      const int ls = r >= G * NP, rl = r - (ls ? G * NP : 0);  // row within its layer's block
      const uint32_t off = r < NR ? (uint32_t)rl * RB + pc * 16 : kOobOff;
      buf[j] = ls ? load16(q1, off) : load16(q0, off);
    }
  };
  load(0);
  for (int r0 = 0; r0 < NR; r0 += R) {
#pragma unroll
    for (int j = 0; j < LPT; ++j) {
      const int i = tid + 256 * j;
      *reinterpret_cast<uint4*>(&tile[(i / NPc) * LDR + (i % NPc) * 8]) = buf[j];
    }
    load(r0 + R);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < R / 16; ++kk) {
      bf16x8_t op[NB];
#pragma unroll
      for (int I = 0; I < NB; ++I) op[I] = gram_operand<LDR>(tile, kk, I, lane);
#pragma unroll
      for (int t = 0; t < NT; ++t)  // block t belongs to wave t / TPW (indices stay compile-time)
        if (t / TPW == wave) acc[t % TPW] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(op[tri.i[t]], op[tri.j[t]], acc[t % TPW], 0, 0, 0);
    }
    __syncthreads();
  }
  float* S = gram_at(P, gs.layer, head);
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    if (t / TPW != wave) continue;
    const int col = 32 * tri.j[t] + (lane & 31);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = 32 * tri.i[t] + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      S[row * D + col] = acc[t % TPW][r];
    }
  }
}

// Gram matrices of D and Dbar over one chunk of kProbeChunk tokens of a
// unit, contracted with S_u, reading the keys once.  64 tokens per step: the
// threads holding a token row's 16-byte pieces of the two layers form its
// fp32 differences, find the token's top-k channels among them
// (row_topk_mask: a bisection over the row's keys with DPP counts), split
// each half difference into bf16 hi + lo (split_bf16x2), zero the top-k
// channels for Dbar, and write the four rows to LDS; waves 0-3 accumulate the
// blocks of D D^T ~ H H^T + H L^T + L H^T (block t on wave t % 4), waves 4-7
// those of Dbar.  Eight waves keep the accumulators at three blocks a wave,
// so four waves fit on a SIMD for the VALU-heavy selection.  The next step's
// loads are in flight during the MFMAs.
template <int D, bool BF16>
__global__ __launch_bounds__(512) void probe_dgram_kernel(ProbeParams P) {
  constexpr int E = BF16 ? 2 : 4;
  constexpr int NPc = D * E / 16;                // 16-byte input pieces per row
  constexpr int CPP = 16 / E;                    // channels per piece
  constexpr int NB = D / 32, NT = NB * (NB + 1) / 2;
  constexpr int WPM = 4, TPW = (NT + WPM - 1) / WPM;  // four waves per matrix: block t on wave t % WPM
  constexpr int R = kGramRows, LDR = D + 16;
  constexpr int LPT = R * NPc / 512;             // loads per thread per layer per step
  // a thread holds PPT pieces of one token row, one from each of its PPT
  // runs of LPR = NPc / PPT pieces (at least 8 lanes, at most 16 keys a lane:
  // fewer count reductions per bisection step of the top-k, more rows per
  // wave, and the LPR lanes' loads of a run are contiguous)
  constexpr int PPT0 = LPT < NPc / 8 ? LPT : NPc / 8;
  constexpr int PPT = PPT0 < 16 / CPP ? PPT0 : 16 / CPP;
  constexpr int LPR = NPc / PPT, KPT = PPT * CPP;
  static_assert(PPT >= 1 && LPT % PPT == 0 && LPR >= 8, "row layout");
  constexpr TriTiles<NB> tri{};
  // [D hi, D lo, Dbar hi, Dbar lo][token][channel]
  __shared__ __attribute__((aligned(16))) uint16_t tile[4][R * LDR];
  __shared__ float red[8];

  const int chunk = blockIdx.x;
  const int bi = blockIdx.y / P.hkv, head = blockIdx.y % P.hkv;
  const int first = P.bl.first[bi];
  const int unit = P.bl.block[bi] * P.hkv + head;
  const int T = P.seq_len, k = P.topk;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const uint64_t RB = (uint64_t)D * E;
  const uint64_t plane = (uint64_t)T * RB;
  const auto ka = make_rsrc(static_cast<const uint8_t*>(P.k[first]) + (uint64_t)head * plane, plane);
  const auto kb = make_rsrc(static_cast<const uint8_t*>(P.k[first + 1]) + (uint64_t)head * plane, plane);
  const int t_begin = chunk * kProbeChunk;
  const int t_end = min(T, t_begin + kProbeChunk);
  const int mat = wave >> 2;                      // 0: D, 1: Dbar

  f32x16_t acc[TPW];
#pragma unroll
  for (int i = 0; i < TPW; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
  // ra[j], rb[j]: piece (j % PPT) LPR + g % LPR of token row g / LPR,
  // g = tid + 512 (j / PPT)
  uint4 ra[LPT], rb[LPT];
  auto load = [&](int t0) {
#pragma unroll
    for (int j = 0; j < LPT; ++j) {
      const int g = tid + 512 * (j / PPT), t = t0 + g / LPR, pc = (j % PPT) * LPR + g % LPR;
      const bool ok = t < t_end;
      ra[j] = load16(ka, ok ? (uint32_t)(t * RB + pc * 16) : kOobOff);
      rb[j] = load16(kb, ok ? (uint32_t)(t * RB + pc * 16) : kOobOff);
    }
  };
  load(t_begin);
  for (int t0 = t_begin; t0 < t_end; t0 += R) {
#pragma unroll
    for (int q = 0; q < LPT / PPT; ++q) {
      const int g = tid + 512 * q, row = g / LPR, lr = g % LPR;
      // the half differences, and the token's top-k keys |fl32(a - b)|: key
      // h CPP + c is channel CPP (h LPR + lr) + c (rows past the chunk read
      // zeros)
      float dv[KPT];
      uint32_t key[KPT];
#pragma unroll
      for (int h = 0; h < PPT; ++h) {
        const uint32_t* pa = reinterpret_cast<const uint32_t*>(&ra[q * PPT + h]);
        const uint32_t* pb = reinterpret_cast<const uint32_t*>(&rb[q * PPT + h]);
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          if constexpr (BF16) {
            const float d0 = bf16_lo(pa[w]) - bf16_lo(pb[w]), d1 = bf16_hi(pa[w]) - bf16_hi(pb[w]);
            key[h * CPP + 2 * w] = as_u32(d0) & 0x7FFFFFFFu;
            key[h * CPP + 2 * w + 1] = as_u32(d1) & 0x7FFFFFFFu;
            dv[h * CPP + 2 * w] = d0 * 0.5f;
            dv[h * CPP + 2 * w + 1] = d1 * 0.5f;
          } else {
            const float d0 = as_f32(pa[w]) - as_f32(pb[w]);
            key[h * CPP + w] = as_u32(d0) & 0x7FFFFFFFu;
            dv[h * CPP + w] = d0 * 0.5f;
          }
        }
      }
      // Dbar: drop the thread's channels that are among the token's top-k
      const uint32_t sel = row_topk_mask<LPR, KPT, PPT>(key, k);
      const uint32_t keep = ~sel & ((1u << KPT) - 1u);
      if (P.ksel) {  // the selection, for compress to reuse
        const int t = t0 + row;
        if (t < t_end)
#pragma unroll
          for (int h = 0; h < PPT; ++h)
            P.ksel[selection_offset(unit, T, t, h * LPR + lr, D, E, P.ksel_bytes)] =
                (uint8_t)((sel >> (h * CPP)) & ((1u << CPP) - 1u));
      }
      uint32_t wd[KPT / 2], wl[KPT / 2], wr[KPT / 2], wrl[KPT / 2];
#pragma unroll
      for (int c = 0; c < KPT / 2; ++c) split_bf16x2(dv[2 * c], dv[2 * c + 1], wd[c], wl[c]);
#pragma unroll
      for (int c = 0; c < KPT / 2; ++c) {
        const uint32_t km = (((keep >> (2 * c)) & 1) ? 0xFFFFu : 0u) | (((keep >> (2 * c + 1)) & 1) ? 0xFFFF0000u : 0u);
        wr[c] = wd[c] & km;
        wrl[c] = wl[c] & km;
      }
      const uint32_t* src[4] = {wd, wl, wr, wrl};
#pragma unroll
      for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int h = 0; h < PPT; ++h) {
          uint16_t* dst = &tile[m][row * LDR + (h * LPR + lr) * CPP];
          const uint32_t* sp = src[m] + h * (CPP / 2);
          if constexpr (CPP == 8)
            *reinterpret_cast<uint4*>(dst) = make_uint4(sp[0], sp[1], sp[2], sp[3]);
          else
            *reinterpret_cast<uint2*>(dst) = make_uint2(sp[0], sp[1]);
        }
    }
    load(t0 + R);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < R / 16; ++kk) {
      bf16x8_t oh[NB], ol[NB];
#pragma unroll
      for (int I = 0; I < NB; ++I) {
        oh[I] = gram_operand<LDR>(tile[2 * mat], kk, I, lane);
        ol[I] = gram_operand<LDR>(tile[2 * mat + 1], kk, I, lane);
      }
#pragma unroll
      for (int t = 0; t < NT; ++t)  // indices stay compile-time
        if (t % WPM == (wave & 3)) {
          const int bi_ = tri.i[t], bj_ = tri.j[t];
          f32x16_t a = __builtin_amdgcn_mfma_f32_32x32x16_bf16(oh[bi_], oh[bj_], acc[t / WPM], 0, 0, 0);
          a = __builtin_amdgcn_mfma_f32_32x32x16_bf16(oh[bi_], ol[bj_], a, 0, 0, 0);
          acc[t / WPM] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ol[bi_], oh[bj_], a, 0, 0, 0);
        }
    }
    __syncthreads();
  }

  // < C, S_u >, off-diagonal blocks counted twice (both matrices symmetric)
  const float* S = gram_at(P, first, head);
  float part = 0.f;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    if (t % WPM != (wave & 3)) continue;
    const float wgt = (tri.i[t] == tri.j[t]) ? 1.f : 2.f;
    const int col = 32 * tri.j[t] + (lane & 31);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = 32 * tri.i[t] + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      part = fmaf(wgt * acc[t / WPM][r], S[row * D + col], part);
    }
  }
  part = wave_sum(part);
  if (lane == 0) red[wave] = part;
  __syncthreads();
  if (tid < 2)
    P.partial[((uint64_t)unit * P.n_chunks + chunk) * 2 + tid] =
        (red[4 * tid] + red[4 * tid + 1]) + (red[4 * tid + 2] + red[4 * tid + 3]);
}

// Blocks of four: Gram matrices of the eight deviation matrices (4 layers x
// shared / residual) over one chunk of kProbeChunk tokens, contracted with
// the layers' probe Gram matrices.  R tokens per step: each thread takes
// one 16-byte piece of a token row from all four layers, forms the
// coefficients Z_1..Z_3 (the fp32 butterfly of dct4.h, as compress ranks
// them), the token's top-k among the row's 3d coefficients with the other
// lanes of the row (row_topk_mask), the block mean, the layer deviations and
// the images of the token's kept coefficients, and writes the eight
// deviation rows to LDS as bf16 hi + lo pairs (split_bf16x2); wave w
// accumulates layer w / 2, shared (w even) or residual (w odd), as
// H H^T + H L^T + L H^T.
template <int D, bool BF16>
__global__ __launch_bounds__(512) void probe_dgram4_kernel(ProbeParams P) {
  constexpr int E = BF16 ? 2 : 4;
  constexpr int NPc = D * E / 16;                // 16-byte input pieces per row
  constexpr int CPP = 16 / E;                    // channels per piece
  constexpr int NB = D / 32, NT = NB * (NB + 1) / 2;
  // LDS rows padded by 16 channels (8 at d = 64, where 16 tiles of 64 rows
  // would pass the 160 KB of a workgroup)
  constexpr int R = 512 / NPc > 32 ? 512 / NPc : 32, LDR = D == 64 ? D + 8 : D + 16;
  constexpr int LPT = R * NPc / 512;             // pieces per thread per step
  constexpr TriTiles<NB> tri{};
  static_assert(LPT >= 1 && R % 16 == 0, "shape");
  // [layer * 2 + residual][hi, lo][token][channel]
  __shared__ __attribute__((aligned(16))) uint16_t tile[16][R * LDR];
  __shared__ float red[8];

  const int chunk = blockIdx.x;
  const int bi = blockIdx.y / P.hkv, head = blockIdx.y % P.hkv;
  const int first = P.bl.first[bi];
  const int unit = P.bl.block[bi] * P.hkv + head;
  const int T = P.seq_len, k = P.topk;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const uint64_t RB = (uint64_t)D * E;
  const uint64_t plane = (uint64_t)T * RB;
  __amdgpu_buffer_rsrc_t kr[4];
#pragma unroll
  for (int n = 0; n < 4; ++n) kr[n] = make_rsrc(static_cast<const uint8_t*>(P.k[first + n]) + (uint64_t)head * plane, plane);
  const int t_begin = chunk * kProbeChunk;
  const int t_end = min(T, t_begin + kProbeChunk);
  const float F1[4] = {kDct4A, kDct4B, -kDct4B, -kDct4A};   // F_4[1][p]
  const float F2[4] = {0.5f, -0.5f, -0.5f, 0.5f};           // F_4[2][p]
  const float F3[4] = {kDct4B, -kDct4A, kDct4A, -kDct4B};   // F_4[3][p]

  f32x16_t acc[NT];
#pragma unroll
  for (int i = 0; i < NT; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
  uint4 rx[LPT][4];
  auto load = [&](int t0) {
#pragma unroll
    for (int j = 0; j < LPT; ++j) {
      const int i = tid + 512 * j, t = t0 + i / NPc, pc = i % NPc;
      const bool ok = t < t_end;
#pragma unroll
      for (int n = 0; n < 4; ++n) rx[j][n] = load16(kr[n], ok ? (uint32_t)(t * RB + pc * 16) : kOobOff);
    }
  };
  load(t_begin);
  for (int t0 = t_begin; t0 < t_end; t0 += R) {
#pragma unroll
    for (int j = 0; j < LPT; ++j) {
      const int i = tid + 512 * j, row = i / NPc, pc = i % NPc;
      // the token's top-k of its 3d coefficients |Z_j[c]|, found by the NPc
      // lanes of its row (rows past the chunk read zeros and add nothing):
      // kept (channel, frequency) pairs of this piece, bit 3 c + j - 1
      uint32_t key[3 * CPP];
#pragma unroll
      for (int c = 0; c < CPP; ++c) {
        float z1, z2, z3;
        dct4_high(chan_of<BF16>(rx[j][0], c), chan_of<BF16>(rx[j][1], c), chan_of<BF16>(rx[j][2], c),
                  chan_of<BF16>(rx[j][3], c), z1, z2, z3);
        key[3 * c] = as_u32(z1) & 0x7FFFFFFFu;
        key[3 * c + 1] = as_u32(z2) & 0x7FFFFFFFu;
        key[3 * c + 2] = as_u32(z3) & 0x7FFFFFFFu;
      }
      const uint32_t kept = row_topk_mask<NPc, 3 * CPP>(key, k);
      if (P.ksel) {  // the selection, for compress to reuse
        const int t = t0 + row;
        if (t < t_end) *reinterpret_cast<uint32_t*>(P.ksel + selection_offset(unit, T, t, pc, D, E, 4)) = kept;
      }
      // the deviations below evaluate the butterfly again rather than keep
      // its 3 CPP results alive beside the accumulators (an empty asm
      // statement that only marks the input pieces as possibly changed)
#pragma unroll
      for (int n = 0; n < 4; ++n) asm volatile("" : "+v"(rx[j][n].x), "+v"(rx[j][n].y), "+v"(rx[j][n].z), "+v"(rx[j][n].w));
      // deviations of the eight matrices, channel pairs at a time, split into bf16 hi + lo
      uint32_t hw[16][CPP / 2];
#pragma unroll
      for (int c2 = 0; c2 < CPP; c2 += 2) {
        float dv[8][2];
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const int c = c2 + e;
          float x[4];
#pragma unroll
          for (int n = 0; n < 4; ++n) x[n] = chan_of<BF16>(rx[j][n], c);
          float z1, z2, z3;  // evaluated again (the same rounded operations): fewer live registers
          dct4_high(x[0], x[1], x[2], x[3], z1, z2, z3);
          const float m = ((x[0] + x[3]) + (x[1] + x[2])) * 0.25f;
          const float k1 = (kept >> (3 * c)) & 1u ? z1 : 0.f;
          const float k2 = (kept >> (3 * c + 1)) & 1u ? z2 : 0.f;
          const float k3 = (kept >> (3 * c + 2)) & 1u ? z3 : 0.f;
#pragma unroll
          for (int n = 0; n < 4; ++n) {
            const float dev = m - x[n];
            dv[2 * n][e] = dev;
            dv[2 * n + 1][e] = dev + (F1[n] * k1 + F2[n] * k2 + F3[n] * k3);
          }
        }
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) split_bf16x2(dv[mt][0], dv[mt][1], hw[2 * mt][c2 >> 1], hw[2 * mt + 1][c2 >> 1]);
      }
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        uint16_t* dst = &tile[m][row * LDR + pc * CPP];
        if constexpr (CPP == 8)
          *reinterpret_cast<uint4*>(dst) = make_uint4(hw[m][0], hw[m][1], hw[m][2], hw[m][3]);
        else
          *reinterpret_cast<uint2*>(dst) = make_uint2(hw[m][0], hw[m][1]);
      }
    }
    load(t0 + R);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < R / 16; ++kk) {
      bf16x8_t oh[NB], ol[NB];
#pragma unroll
      for (int I = 0; I < NB; ++I) {
        oh[I] = gram_operand<LDR>(tile[2 * wave], kk, I, lane);
        ol[I] = gram_operand<LDR>(tile[2 * wave + 1], kk, I, lane);
      }
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        f32x16_t a = __builtin_amdgcn_mfma_f32_32x32x16_bf16(oh[tri.i[t]], oh[tri.j[t]], acc[t], 0, 0, 0);
        a = __builtin_amdgcn_mfma_f32_32x32x16_bf16(oh[tri.i[t]], ol[tri.j[t]], a, 0, 0, 0);
        acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ol[tri.i[t]], oh[tri.j[t]], a, 0, 0, 0);
      }
    }
    __syncthreads();
  }

  // < C, S_p >, off-diagonal blocks counted twice (both matrices symmetric)
  const float* S = gram_at(P, first + (wave >> 1), head);
  float part = 0.f;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const float wgt = (tri.i[t] == tri.j[t]) ? 1.f : 2.f;
    const int col = 32 * tri.j[t] + (lane & 31);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = 32 * tri.i[t] + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      part = fmaf(wgt * acc[t][r], S[row * D + col], part);
    }
  }
  part = wave_sum(part);
  if (lane == 0) red[wave] = part;
  __syncthreads();
  if (tid < 2)
    P.partial[((uint64_t)unit * P.n_chunks + chunk) * 2 + tid] = (red[tid] + red[2 + tid]) + (red[4 + tid] + red[6 + tid]);
}

__global__ void probe_finalize_kernel(ProbeParams P) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int units = P.n_blocks * P.hkv;
  if (i >= units * 2) return;
  const int unit = i >> 1, m = i & 1;
  double s = 0.0;
  for (int c = 0; c < P.n_chunks; ++c) s += (double)P.partial[((uint64_t)unit * P.n_chunks + c) * 2 + m];
  const int G = P.hq / P.hkv;
  const double nl = (double)P.bsizes[unit / P.hkv];
  P.errors[unit * 2 + m] = (float)(s / (nl * G * (double)P.n_probe * (double)P.d));
}

template <int D, bool BF16>
static hipError_t launch_probe_t(const ProbeParams& P, hipStream_t s) {
  const int slots = P.bl.n * P.hkv * (P.bsize == 2 ? 1 : 4);
  if constexpr (BF16)
    hipLaunchKernelGGL((probe_qgram_mfma_kernel<D>), dim3(slots), dim3(256), 0, s, P);
  else
    hipLaunchKernelGGL((probe_qgram_kernel<D, BF16>), dim3(slots), dim3(256), 0, s, P);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 grid(P.n_chunks, P.bl.n * P.hkv);
  if (P.bsize == 4)
    hipLaunchKernelGGL((probe_dgram4_kernel<D, BF16>), grid, dim3(512), 0, s, P);
  else
    hipLaunchKernelGGL((probe_dgram_kernel<D, BF16>), grid, dim3(512), 0, s, P);
  return hipGetLastError();
}

hipError_t launch_probe(const ProbeParams& P, hipStream_t s) {
  if (P.bl.n == 0) return hipSuccess;
  if (P.d == 128) return P.bf16 ? launch_probe_t<128, true>(P, s) : launch_probe_t<128, false>(P, s);
  return P.bf16 ? launch_probe_t<64, true>(P, s) : launch_probe_t<64, false>(P, s);
}

hipError_t launch_probe_finalize(const ProbeParams& P, hipStream_t s) {
  const int units = P.n_blocks * P.hkv;
  hipLaunchKernelGGL(probe_finalize_kernel, dim3((units * 2 + 255) / 256), dim3(256), 0, s, P);
  return hipGetLastError();
}

}  // namespace fdkv
