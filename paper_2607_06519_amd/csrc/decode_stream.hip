// Streaming split-K decode over a bf16 compressed cache (Section 3, the
// reconstruction fused into attention after Eq. 3).
//
// One workgroup = 4 waves = 512 tokens of one (sequence, KV head); a wave
// walks its 128 tokens in 16-row tiles with an online softmax and keeps the
// next tile's loads in flight while it computes the current one (two
// register buffers).
//
// Lane layout (the same for K and V): NP = d/8 lanes per row, lane holds one
// 16-byte piece (8 bf16 channels); a load instruction covers RPV = 64/NP
// consecutive rows (1 KB, fully coalesced).  Loads are raw buffer loads
// (32-bit offsets, SGPR descriptors); rows past the sequence end read as 0.
//
// Per tile:
//  K  - bf16 dot2 of the lane's piece with the matching query piece, group
//       sum over the NP lanes of the row by DPP; residual heads add
//       sigma * q[IK_j] * D_K,j for the lane's residual entry.
//  softmax - against a running reference max that moves (wave max, rescale
//       by exp2(m_old - m_new)) only when a logit exceeds it by more than
//       2^8; probabilities to LDS (fp32 and bf16 pairs).
//  V  - rows r and r + RPV are paired so one dot2 multiplies two tokens'
//       values by their two bf16 probabilities; residual V entries are added
//       into LDS accumulators (one copy per row slot r % 4, so the lanes of a
//       step never collide), rescaled together with the rest.
// The 4 waves merge in LDS and write one (acc, m, l) record per workgroup;
// decode_merge combines the records.  HBM bound: no MFMA.
#include "fdkv_common.h"
#include "fdkv_kernels.h"

namespace fdkv {

namespace {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
constexpr int kRsrcDword3 = 0x00020000;  // raw buffer, 32-bit data format (gfx9 family)
constexpr float kSlack = 8.f;            // log2 headroom of the running reference max

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), c,
                                         false);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, uint64_t bytes) {
  const uint32_t n = bytes > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, kRsrcDword3);
}

__device__ __forceinline__ uint4 ld128(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

template <int D, int G>
struct SS {
  static constexpr int NP = D / 8;                 // 16-byte pieces per bf16 row
  static constexpr int CPP = 8;                    // channels per piece
  // K pass: LPRK lanes per row, PKK pieces per lane, RSK rows per load set
  static constexpr int LPRK = (G >= 8 || NP < 8) ? (NP < 8 ? NP : 8) : 4;
  static constexpr int PKK = NP / LPRK;
  static constexpr int RSK = 64 / LPRK;
  // V pass: NP lanes per row (one piece each), RPL rows per load
  static constexpr int RPL = 64 / NP;
  static constexpr int TILE = 16;
  static constexpr int NKS = TILE / RSK;           // K load sets per tile
  static constexpr int NL = TILE / RPL;            // V loads per tile
  static constexpr int NPAIR = NL / 2;
  static constexpr int CW = kDecodeChunk;          // tokens per wave
  static constexpr int NT = CW / TILE;
  static constexpr int KEL = 16 / LPRK;            // residual K entries per lane per row (k = 16 path)
  static constexpr int W = kDecodeWaves;
  static constexpr int RS = D + 4;
  static_assert(NKS >= 1 && NL % 2 == 0 && NT % 2 == 0 && TILE * 16 == 64 * 4, "shape");
};

template <int D, int G>
struct TileBuf {
  using S = SS<D, G>;
  uint4 k[S::NKS][S::PKK];
  uint4 v[S::NL];
  uint32_t ki[S::NKS];            // residual K indices of the lane's entries (k = 16 path)
  uint32_t kv[S::NKS][2];         // their bf16 values
  uint32_t vi[4];                 // residual V index of the lane in each 4-row step (k = 16 path)
  uint32_t vv[4];                 // its bf16 value
};

}  // namespace

template <int D, int G>
__global__ __launch_bounds__(256) void decode_stream_kernel(DecodeParams P) {
  using S = SS<D, G>;
  constexpr int NP = S::NP, CPP = S::CPP, LPRK = S::LPRK, PKK = S::PKK, RSK = S::RSK, RPL = S::RPL;
  constexpr int TILE = S::TILE, NKS = S::NKS, NL = S::NL, NPAIR = S::NPAIR, CW = S::CW, NT = S::NT;
  constexpr int KEL = S::KEL, W = S::W;
  constexpr uint32_t RB = D * 2;
  __shared__ float q_lds[D * G];               // [c][g] fp32, residual K gathers
  __shared__ uint4 qp_lds[G][NP];              // bf16 query pieces for the K pass
  __shared__ uint32_t pp_lds[W][G][TILE / 2];  // bf16 probability pairs of the tile
  __shared__ float p_lds[W][G][TILE];          // fp32 probabilities of the tile
  __shared__ float sp_lds[W][4][G][D];         // residual V accumulator, one copy per row slot r % 4
  __shared__ float mg_lds[W][G][D + 2];        // per-wave acc, m, l

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wgc = blockIdx.x % P.n_wgchunks;
  const int sh = blockIdx.x / P.n_wgchunks;
  const int head = sh % P.hkv, seq = sh / P.hkv;
  const int T = P.seq_lens[seq];
  const int wg_tok0 = wgc * kDecodeWgTokens;
  if (wg_tok0 >= T) return;

  const int pair = P.layer >> 1, parity = P.layer & 1;
  const float sigma = parity ? -1.f : 1.f;
  const uint64_t unit = ((uint64_t)seq * P.n_pairs + pair) * P.hkv + head;
  const int mode = P.modes[unit];
  const int k = P.topk;
  const bool resid = (mode == kResidual) && k > 0;
  const bool resid16 = resid && k == 16 && NP == 16;
  const uint8_t* seg = P.cache + P.seg_off[unit];
  const SegLayout L = seg_layout(mode, (uint64_t)T, D, k, 2);
  const uint64_t dense = (uint64_t)T * RB;
  const auto kr = rsrc(seg + (mode == kExact ? (parity ? L.k1 : L.k0) : L.mk), dense);
  const auto vr = rsrc(seg + (mode == kExact ? (parity ? L.v1 : L.v0) : L.mv), dense);
  const auto ikr = rsrc(seg + L.ik, (uint64_t)T * k);
  const auto vkr = rsrc(seg + L.vk, (uint64_t)T * k * 2);
  const auto ivr = rsrc(seg + L.iv, (uint64_t)T * k);
  const auto vvr = rsrc(seg + L.vv, (uint64_t)T * k * 2);
  const uint8_t* qbase = static_cast<const uint8_t*>(P.q) + ((uint64_t)seq * P.hq + (uint64_t)head * G) * RB;

  for (int i = threadIdx.x; i < D * G; i += 256) {
    const int g = i / D, c = i % D;
    q_lds[c * G + g] = bf16_to_f32(reinterpret_cast<const uint16_t*>(qbase)[g * D + c]);
  }
  for (int i = lane; i < 4 * G * D; i += 64) (&sp_lds[wave][0][0][0])[i] = 0.f;

  const int krow = lane / LPRK, ks = lane % LPRK;  // K pass: row in load set, lane in row
  const int rr = lane / NP, pc = lane % NP;        // V pass: row in load, piece
  for (int i = threadIdx.x; i < G * NP; i += 256)
    qp_lds[i / NP][i % NP] = *reinterpret_cast<const uint4*>(qbase + (uint64_t)(i / NP) * RB + (uint64_t)(i % NP) * 16);
  __syncthreads();

  const int wtok0 = wg_tok0 + wave * CW;
  const int ntiles = wtok0 < T ? min(NT, (T - wtok0 + TILE - 1) / TILE) : 0;

  float m[G], l[G], acc[G][CPP];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -INFINITY;
    l[g] = 0.f;
#pragma unroll
    for (int c = 0; c < CPP; ++c) acc[g][c] = 0.f;
  }

  auto load = [&](int t, TileBuf<D, G>& b) {
    const uint32_t r0 = (uint32_t)(wtok0 + t * TILE);
#pragma unroll
    for (int ks_ = 0; ks_ < NKS; ++ks_) {
      const uint32_t row = r0 + ks_ * RSK + krow;
#pragma unroll
      for (int j = 0; j < PKK; ++j) b.k[ks_][j] = ld128(kr, row * RB + (uint32_t)(j * LPRK + ks) * 16);
      if (resid16) {
        const uint32_t e = row * 16 + ks * KEL;
        if constexpr (KEL == 4) {
          b.ki[ks_] = __builtin_amdgcn_raw_buffer_load_b32(ikr, e, 0, 0);
          const auto w2 = __builtin_amdgcn_raw_buffer_load_b64(vkr, e * 2, 0, 0);
          b.kv[ks_][0] = w2[0];
          b.kv[ks_][1] = w2[1];
        } else {
          b.ki[ks_] = __builtin_amdgcn_raw_buffer_load_b16(ikr, e, 0, 0);
          b.kv[ks_][0] = __builtin_amdgcn_raw_buffer_load_b32(vkr, e * 2, 0, 0);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < NL; ++i) b.v[i] = ld128(vr, (r0 + i * RPL + rr) * RB + pc * 16);
    if (resid16) {
      // step jj covers rows 4jj..4jj+3 of the tile: lane = (row slot lane / 16, entry lane % 16)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const uint32_t e = (r0 + 4 * jj + (lane >> 4)) * 16 + (lane & 15);
        b.vi[jj] = __builtin_amdgcn_raw_buffer_load_b8(ivr, e, 0, 0);
        b.vv[jj] = __builtin_amdgcn_raw_buffer_load_b16(vvr, e * 2, 0, 0);
      }
    }
  };

  auto compute = [&](int t, const TileBuf<D, G>& b) {
    const int r0 = wtok0 + t * TILE;
    float s[NKS][G];
#pragma unroll
    for (int ks_ = 0; ks_ < NKS; ++ks_) {
      float a[G];
#pragma unroll
      for (int g = 0; g < G; ++g) a[g] = 0.f;
#pragma unroll
      for (int j = 0; j < PKK; ++j) {
        const uint32_t* kw = reinterpret_cast<const uint32_t*>(&b.k[ks_][j]);
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const uint4 qv = qp_lds[g][j * LPRK + ks];
          const uint32_t* qw = reinterpret_cast<const uint32_t*>(&qv);
#pragma unroll
          for (int w = 0; w < 4; ++w) a[g] = dot2(kw[w], qw[w], a[g]);
        }
      }
      const int row = r0 + ks_ * RSK + krow;
      if (resid16) {
#pragma unroll
        for (int e = 0; e < KEL; ++e) {
          const int c = (b.ki[ks_] >> (8 * e)) & (D - 1);
          const float v = sigma * bf16_to_f32((uint16_t)(b.kv[ks_][e >> 1] >> (16 * (e & 1))));
#pragma unroll
          for (int g = 0; g < G; ++g) a[g] = fmaf(q_lds[c * G + g], v, a[g]);
        }
      } else if (resid) {
        const uint32_t rc = (uint32_t)min(row, T - 1);
        for (int e = ks; e < k; e += LPRK) {
          const int c = __builtin_amdgcn_raw_buffer_load_b8(ikr, rc * k + e, 0, 0) & (D - 1);
          const float v =
              sigma * bf16_to_f32((uint16_t)__builtin_amdgcn_raw_buffer_load_b16(vkr, (rc * k + e) * 2, 0, 0));
#pragma unroll
          for (int g = 0; g < G; ++g) a[g] = fmaf(q_lds[c * G + g], v, a[g]);
        }
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float x = group_sum<LPRK>(a[g]) * P.scale_log2;
        s[ks_][g] = row < T ? x : -INFINITY;
      }
    }
    // online softmax over the tile.  m is a reference value, uniform over the
    // wave, that only moves when some logit exceeds it by more than kSlack
    // (probabilities then stay below 2^kSlack); moving it takes a wave max
    // and rescales the running sums.
    bool rescale = false;
    float alpha[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float mt = s[0][g];
#pragma unroll
      for (int ks_ = 1; ks_ < NKS; ++ks_) mt = fmaxf(mt, s[ks_][g]);
      float mn = m[g];
      alpha[g] = 1.f;
      if (__ballot(mt > m[g] + kSlack) != 0) {
#pragma unroll
        for (int o = LPRK; o < 64; o <<= 1) mt = fmaxf(mt, __shfl_xor(mt, o, 64));
        mn = fmaxf(m[g], mt);
        alpha[g] = (m[g] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m[g] - mn);
        rescale = true;
      }
      float ps = 0.f;
#pragma unroll
      for (int ks_ = 0; ks_ < NKS; ++ks_) {
        const float p = (s[ks_][g] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(s[ks_][g] - mn);
        ps += p;
        if (ks == 0) {
          const int R = ks_ * RSK + krow;  // tile-local row; rows R and R + RPL share a pair slot
          const int i = R / RPL;
          p_lds[wave][g][R] = p;
          reinterpret_cast<uint16_t*>(&pp_lds[wave][g][0])[((i >> 1) * RPL + R % RPL) * 2 + (i & 1)] =
              (uint16_t)f32_to_bf16_bits(p);
        }
      }
      l[g] = l[g] * alpha[g] + (ks == 0 ? ps : 0.f);
      m[g] = mn;
    }
    if (rescale) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
#pragma unroll
        for (int c = 0; c < CPP; ++c) acc[g][c] *= alpha[g];
        if (resid) {
#pragma unroll
          for (int cp = 0; cp < 4; ++cp)
#pragma unroll
            for (int c = lane; c < D; c += 64) sp_lds[wave][cp][g][c] *= alpha[g];
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // P V over the dense plane
#pragma unroll
    for (int pr = 0; pr < NPAIR; ++pr) {
      uint32_t pp[G];
#pragma unroll
      for (int g = 0; g < G; ++g) pp[g] = pp_lds[wave][g][pr * RPL + rr];
      const uint32_t* wa = reinterpret_cast<const uint32_t*>(&b.v[2 * pr]);
      const uint32_t* wb = reinterpret_cast<const uint32_t*>(&b.v[2 * pr + 1]);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint32_t lo = __builtin_amdgcn_perm(wb[w], wa[w], 0x05040100u);
        const uint32_t hi = __builtin_amdgcn_perm(wb[w], wa[w], 0x07060302u);
#pragma unroll
        for (int g = 0; g < G; ++g) {
          acc[g][2 * w] = dot2(lo, pp[g], acc[g][2 * w]);
          acc[g][2 * w + 1] = dot2(hi, pp[g], acc[g][2 * w + 1]);
        }
      }
    }
    // residual V entries.  In one step the lanes touch 4 rows (one accumulator
    // copy each) and the 16 distinct channels of each row, so no two lanes of
    // an LDS instruction share an address and a plain read-add-write is exact.
    if (resid16) {
      const int slot = lane >> 4;
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int rl = 4 * jj + slot;
        if (r0 + rl < T) {
          const int c = b.vi[jj] & (D - 1);
          const float v = sigma * bf16_to_f32((uint16_t)b.vv[jj]);
#pragma unroll
          for (int g = 0; g < G; ++g) sp_lds[wave][slot][g][c] += p_lds[wave][g][rl] * v;
        }
      }
    } else if (resid) {
      for (int ent = lane; ent < TILE * k; ent += 64) {
        const int rl = ent / k;
        if (r0 + rl < T) {
          const uint32_t ix = (uint32_t)(r0 + rl) * k + (ent - rl * k);
          const int c = __builtin_amdgcn_raw_buffer_load_b8(ivr, ix, 0, 0) & (D - 1);
          const float v = sigma * bf16_to_f32((uint16_t)__builtin_amdgcn_raw_buffer_load_b16(vvr, ix * 2, 0, 0));
#pragma unroll
          for (int g = 0; g < G; ++g) atomicAdd(&sp_lds[wave][0][g][c], p_lds[wave][g][rl] * v);
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };

  if (ntiles > 0) {
    TileBuf<D, G> A, Bf;
    load(0, A);
    for (int t = 0; t < ntiles; t += 2) {
      if (t + 1 < ntiles) load(t + 1, Bf);
      compute(t, A);
      if (t + 1 < ntiles) {
        if (t + 2 < ntiles) load(t + 2, A);
        compute(t + 1, Bf);
      }
    }
  }

  // wave totals
#pragma unroll
  for (int g = 0; g < G; ++g) l[g] = wave_sum(l[g]);
#pragma unroll
  for (int o = NP; o < 64; o <<= 1)
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int c = 0; c < CPP; ++c) acc[g][c] += __shfl_xor(acc[g][c], o, 64);
  __syncthreads();
  if (lane < NP) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int c = 0; c < CPP; ++c)
        mg_lds[wave][g][lane * CPP + c] = acc[g][c] + sp_lds[wave][0][g][lane * CPP + c] +
                                          sp_lds[wave][1][g][lane * CPP + c] + sp_lds[wave][2][g][lane * CPP + c] +
                                          sp_lds[wave][3][g][lane * CPP + c];
  }
  if (lane == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      mg_lds[wave][g][D] = m[g];
      mg_lds[wave][g][D + 1] = l[g];
    }
  }
  __syncthreads();
  float* rec = P.ws + ((uint64_t)sh * P.n_wgchunks + wgc) * G * S::RS;
  for (int i = threadIdx.x; i < G * (D + 2); i += 256) {
    const int g = i / (D + 2), c = i - g * (D + 2);
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < W; ++w) M = fmaxf(M, mg_lds[w][g][D]);
    float o;
    if (c == D) {
      o = M;
    } else {
      o = 0.f;
#pragma unroll
      for (int w = 0; w < W; ++w) {
        const float mw = mg_lds[w][g][D];
        const float f = (mw == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mw - M);
        o = fmaf(f, mg_lds[w][g][c], o);
      }
    }
    rec[g * S::RS + c] = o;
  }
}

// Log-sum-exp merge of the workgroup records of one (sequence, query head):
//   M = max_i m_i,  l = sum_i l_i 2^(m_i - M),  o = sum_i acc_i 2^(m_i - M) / l.
// One 512-thread workgroup per query head; records are taken in blocks of
// 512, the channels split over 512 / d thread groups that each sum a strided
// subset of the block's records.
template <int D, bool BF16, int G>
__global__ __launch_bounds__(512) void decode_merge_kernel(DecodeParams P) {
  constexpr int RS = D + 4;
  constexpr int NB = 512;            // records per block
  constexpr int SUB = 512 / D;       // thread groups per channel
  __shared__ float wgt[NB];
  __shared__ float red[512];
  __shared__ float part[SUB][D];
  const int qh = blockIdx.x % P.hq, seq = blockIdx.x / P.hq;
  const int head = qh / G, g = qh % G;
  const int T = P.seq_lens[seq];
  const int nch = min((T + kDecodeWgTokens - 1) / kDecodeWgTokens, P.n_wgchunks);
  const float* base = P.ws + ((uint64_t)(seq * P.hkv + head) * P.n_wgchunks) * G * RS + g * RS;
  const int tid = threadIdx.x;
  const int c = tid % D, sub = tid / D;
  float M = -INFINITY, Lsum = 0.f, acc = 0.f;
  for (int b0 = 0; b0 < nch; b0 += NB) {
    const int nb = min(NB, nch - b0);
    const float mi = tid < nb ? base[(uint64_t)(b0 + tid) * G * RS + D] : -INFINITY;
    red[tid] = mi;
    __syncthreads();
    for (int o = 256; o > 0; o >>= 1) {
      if (tid < o) red[tid] = fmaxf(red[tid], red[tid + o]);
      __syncthreads();
    }
    const float Mb = red[0];
    __syncthreads();
    const float wi = tid < nb ? __builtin_amdgcn_exp2f(mi - Mb) : 0.f;
    wgt[tid] = wi;
    red[tid] = tid < nb ? wi * base[(uint64_t)(b0 + tid) * G * RS + D + 1] : 0.f;
    __syncthreads();
    for (int o = 256; o > 0; o >>= 1) {
      if (tid < o) red[tid] += red[tid + o];
      __syncthreads();
    }
    const float Lb = red[0];
    float ab = 0.f;
#pragma unroll 8
    for (int i = sub; i < nb; i += SUB) ab = fmaf(wgt[i], base[(uint64_t)(b0 + i) * G * RS + c], ab);
    part[sub][c] = ab;
    __syncthreads();
    if (sub == 0) {
#pragma unroll
      for (int j = 1; j < SUB; ++j) ab += part[j][c];
    }
    // fold the block into the running result (rescale by the new max)
    const float Mn = fmaxf(M, Mb);
    const float fo = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(M - Mn);
    const float fb = __builtin_amdgcn_exp2f(Mb - Mn);
    Lsum = Lsum * fo + Lb * fb;
    acc = acc * fo + ab * fb;
    M = Mn;
    __syncthreads();
  }
  if (sub == 0) {
    const float res = nch > 0 ? acc / Lsum : 0.f;
    const uint64_t oi = ((uint64_t)seq * P.hq + qh) * D + c;
    if constexpr (BF16)
      reinterpret_cast<uint16_t*>(P.out)[oi] = (uint16_t)f32_to_bf16_bits(res);
    else
      reinterpret_cast<float*>(P.out)[oi] = res;
  }
}

template <int D, int G>
static hipError_t launch_t(const DecodeParams& P, hipStream_t s) {
  const unsigned nsh = (unsigned)P.batch * P.hkv;
  hipLaunchKernelGGL((decode_stream_kernel<D, G>), dim3(nsh * P.n_wgchunks), dim3(256), 0, s, P);
  return hipGetLastError();
}

hipError_t launch_decode_stream(const DecodeParams& P, hipStream_t s) {
  if (P.n_wgchunks <= 0) return hipSuccess;
  const int G = P.hq / P.hkv;
  if (P.d == 128) {
    switch (G) {
      case 1: return launch_t<128, 1>(P, s);
      case 2: return launch_t<128, 2>(P, s);
      case 4: return launch_t<128, 4>(P, s);
      default: return launch_t<128, 8>(P, s);
    }
  }
  switch (G) {
    case 1: return launch_t<64, 1>(P, s);
    case 2: return launch_t<64, 2>(P, s);
    case 4: return launch_t<64, 4>(P, s);
    default: return launch_t<64, 8>(P, s);
  }
}

template <int D, bool BF16>
static hipError_t launch_merge_d(const DecodeParams& P, hipStream_t s) {
  const dim3 grid((unsigned)P.batch * P.hq);
  switch (P.hq / P.hkv) {
    case 1: hipLaunchKernelGGL((decode_merge_kernel<D, BF16, 1>), grid, dim3(512), 0, s, P); break;
    case 2: hipLaunchKernelGGL((decode_merge_kernel<D, BF16, 2>), grid, dim3(512), 0, s, P); break;
    case 4: hipLaunchKernelGGL((decode_merge_kernel<D, BF16, 4>), grid, dim3(512), 0, s, P); break;
    default: hipLaunchKernelGGL((decode_merge_kernel<D, BF16, 8>), grid, dim3(512), 0, s, P); break;
  }
  return hipGetLastError();
}

hipError_t launch_decode_merge(const DecodeParams& P, hipStream_t s) {
  if (P.d == 128) return P.bf16 ? launch_merge_d<128, true>(P, s) : launch_merge_d<128, false>(P, s);
  return P.bf16 ? launch_merge_d<64, true>(P, s) : launch_merge_d<64, false>(P, s);
}

}  // namespace fdkv
