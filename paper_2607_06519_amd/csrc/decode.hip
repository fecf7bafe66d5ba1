// Decode attention over the compressed cache with the reconstruction fused
// in (Section 3, the paragraph after Eq. 3): shared coefficients are read once
// per token and the sparse residual is added only at its indexed channels;
// no reconstructed K/V is ever materialised.
//
// For layer p of a block of B layers and the G query heads of a KV head:
//   shared   : K~ = MK,                             V~ = MV
//   residual : K~ = MK + sum_e w_e value_e at c_e,  V~ likewise
//   exact    : K~ = K_p,                            V~ = V_p
// where an entry e is a channel c_e with w_e = +1 (p = 0) or -1 (p = 1) for
// the stored half difference of a pair, or a code 4c_e + j with
// w_e = F_4[j][p] for a block of four.  Logits use the algebraic form
// q.K~ = q.MK + sum_e w_e q[c_e] value_e.
//
// decode_splitk (the fp32 cache path; bf16 caches use decode_stream.hip): one
// workgroup = 4 waves = 512 tokens of one (sequence, KV head); each wave
// takes 128 tokens in two passes over HBM-resident planes:
//   K pass - 4 (G <= 4) or 8 lanes per row read 16-byte pieces; bf16 dot2
//            against the query pieces held in registers, group reduction by
//            DPP; logits (log2 domain) to LDS.
//   V pass - one row per NP lanes, rows paired so that two tokens' bf16
//            values and their bf16 probabilities form one dot2; the sparse
//            V residual goes into an LDS accumulator with ds_add_f32.
// The chunk max is exact (two passes), so no rescaling is needed inside a
// wave; the 4 waves merge in LDS and the workgroup writes one (acc, m, l)
// record.  decode_merge (decode_stream.hip) merges the records of a
// sequence with the log-sum-exp rule.
#include "fdkv_common.h"
#include "fdkv_kernels.h"

namespace fdkv {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), c,
                                         false);
}

template <int D, bool BF16, int G>
struct DecodeShape {
  static constexpr int E = BF16 ? 2 : 4;
  static constexpr int NP = D * E / 16;          // 16-byte pieces per row
  static constexpr int CPP = 16 / E;             // channels per piece
  static constexpr int LPRK = (G >= 8) ? 8 : 4;  // lanes per row in the K pass
  static constexpr int PK = NP / LPRK;           // pieces per lane in the K pass
  static constexpr int RPK = 64 / LPRK;          // rows per K pass step
  static constexpr int RPV = 64 / NP;            // rows per V load
  static constexpr int CH = kDecodeChunk;
  static constexpr int W = kDecodeWaves;
  static constexpr int RS = D + 4;               // partial record stride (floats)
  static_assert(PK >= 1 && CH % RPK == 0 && CH % (2 * RPV) == 0 && CH % 64 == 0, "shape");
};

template <int D, bool BF16>
__device__ __forceinline__ float load_elem(const uint8_t* base, uint64_t i) {
  if constexpr (BF16)
    return bf16_to_f32(reinterpret_cast<const uint16_t*>(base)[i]);
  else
    return reinterpret_cast<const float*>(base)[i];
}

template <int D, bool BF16, int G>
__global__ __launch_bounds__(256) void decode_splitk_kernel(DecodeParams P) {
  using S = DecodeShape<D, BF16, G>;
  constexpr int E = S::E, NP = S::NP, CPP = S::CPP, LPRK = S::LPRK, PK = S::PK;
  constexpr int RPK = S::RPK, RPV = S::RPV, CH = S::CH, W = S::W;
  __shared__ float q_lds[D * G];            // [c][g], for residual gathers
  __shared__ float s_lds[W][G][CH];         // logits, then probabilities
  __shared__ uint32_t pp_lds[W][G][CH / 2]; // bf16 probability pairs (rows r, r + RPV)
  __shared__ float sp_lds[W][G][D];         // sparse V accumulator
  __shared__ float mg_lds[W][G][D + 2];     // per-wave acc, m, l

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int slot = blockIdx.x % P.n_chunks_total;
  const int sh = blockIdx.x / P.n_chunks_total;  // seq * hkv + head
  const int head = sh % P.hkv, seq = sh / P.hkv;
  const int part = decode_part(P, slot);
  const int wgc = slot - P.part[part].base;
  const bool tail = part == P.tail_part;
  const int T = P.part[part].lens[seq];
  const int wg_tok0 = wgc * kDecodeWgTokens;
  const uint64_t unit = ((uint64_t)seq * P.n_blocks + P.block) * P.hkv + head;
  // the exact tail of a generation has no unit arrays
  const uint32_t mbyte = tail ? (uint32_t)kExact : P.part[part].modes[unit];
  const int mode = mode_of(mbyte);
  const uint64_t seg_off = tail ? 0 : P.part[part].seg_off[unit];
  const bool bad_unit = !unit_byte_ok(mbyte, P.tokres ? P.n_rates : 0) || (seg_off & 255) != 0;
  if (wg_tok0 >= T || bad_unit) {  // uniform over the workgroup
    // an empty record (m = -inf, l = 0, acc = 0): the merge reads every slot;
    // an invalid unit (mode above exact or a misaligned segment) writes
    // m = 0, l = 1, acc = NaN, which turns its query heads' outputs into NaN
    float* rec = P.ws + ((uint64_t)sh * P.n_chunks_total + slot) * G * S::RS;
    for (int i = threadIdx.x; i < G * S::RS; i += 256) {
      const int c = i % S::RS;
      rec[i] = bad_unit ? (c == D ? 0.f : c == D + 1 ? 1.f : __builtin_nanf("")) : (c == D ? -INFINITY : 0.f);
    }
    return;
  }

  const bool q4 = P.bsize == 4;
  const int k = P.topk;
  const bool resid = !P.tokres && (mode == kResidual) && k > 0;
  const bool tokres = P.tokres && mode == kResidual;   // token-level residual set
  const uint8_t* seg = tail ? static_cast<const uint8_t*>(P.tail_k) : P.part[part].cache + seg_off;
  const SegLayout L = seg_layout(mode, (uint64_t)T, D, k, E, E, P.bsize);
  const uint64_t xplane = plane_bytes((uint64_t)T * D * E);  // exact planes: K_p at p * xplane, V_p at (B + p) * xplane
  const uint64_t tail_off = ((uint64_t)seq * P.hkv + head) * (uint64_t)P.tail_cap * D * E;
  const uint8_t* kplane = tail ? static_cast<const uint8_t*>(P.tail_k) + tail_off
                               : seg + (mode == kExact ? (uint64_t)P.pos * xplane : L.mk);
  const uint8_t* vplane = tail ? static_cast<const uint8_t*>(P.tail_v) + tail_off
                               : seg + (mode == kExact ? (uint64_t)(P.bsize + P.pos) * xplane : L.mv);
  // channel and weight of residual entry i of an index plane
  auto entry = [&](const uint8_t* ip, uint64_t i, float& w) -> int {
    if (q4) {
      const uint32_t code = reinterpret_cast<const uint16_t*>(ip)[i];
      const uint32_t j = code & 3u;
      const uint32_t m1 = 0u - (uint32_t)(j == 1u), m2 = 0u - (uint32_t)(j == 2u), m3 = 0u - (uint32_t)(j == 3u);
      w = as_f32((as_u32(P.wres[0]) & m1) | (as_u32(P.wres[1]) & m2) | (as_u32(P.wres[2]) & m3));
      return (int)(code >> 2) & (D - 1);
    }
    w = P.wres[0];
    return ip[i] & (D - 1);
  };
  const uint8_t* ikp = seg + L.ik;
  const uint8_t* vkp = seg + L.vk;
  const uint8_t* ivp = seg + L.iv;
  const uint8_t* vvp = seg + L.vv;
  const uint8_t* qbase = static_cast<const uint8_t*>(P.q) + ((uint64_t)seq * P.hq + (uint64_t)head * G) * D * E;
  const uint64_t RB = (uint64_t)D * E;

  for (int i = threadIdx.x; i < D * G; i += 256) {
    const int g = i / D, c = i % D;
    q_lds[c * G + g] = load_elem<D, BF16>(qbase, (uint64_t)g * D + c);
  }
  for (int i = lane; i < G * D; i += 64) (&sp_lds[wave][0][0])[i] = 0.f;

  const int kr = lane / LPRK, ks = lane % LPRK;
  uint4 qr[G][PK];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int j = 0; j < PK; ++j)
      qr[g][j] = *reinterpret_cast<const uint4*>(qbase + (uint64_t)g * RB + (uint64_t)(j * LPRK + ks) * 16);
  __syncthreads();

  const int wtok0 = wg_tok0 + wave * CH;

  // ------------------------------------------------------------ K pass
  float mx[G];
#pragma unroll
  for (int g = 0; g < G; ++g) mx[g] = -INFINITY;
  const int epl = (k + LPRK - 1) / LPRK;
  const int e0 = ks * epl, e1 = min(k, e0 + epl);
  for (int pass = 0; pass < CH / RPK; ++pass) {
    const int row = wtok0 + pass * RPK + kr;
    const int rc = min(row, T - 1);
    const uint4* src = reinterpret_cast<const uint4*>(kplane + (uint64_t)rc * RB);
    uint4 kv[PK];
#pragma unroll
    for (int j = 0; j < PK; ++j) kv[j] = src[j * LPRK + ks];
    float a[G];
#pragma unroll
    for (int g = 0; g < G; ++g) a[g] = 0.f;
#pragma unroll
    for (int j = 0; j < PK; ++j) {
      const uint32_t* kw = reinterpret_cast<const uint32_t*>(&kv[j]);
#pragma unroll
      for (int w = 0; w < 4; ++w)
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const uint32_t qw = reinterpret_cast<const uint32_t*>(&qr[g][j])[w];
          if constexpr (BF16)
            a[g] = dot2_bf16(kw[w], qw, a[g]);
          else
            a[g] = fmaf(as_f32(kw[w]), as_f32(qw), a[g]);
        }
    }
    if (resid) {
      for (int e = e0; e < e1; ++e) {
        float w;
        const int c = entry(ikp, (uint64_t)rc * k + e, w);
        const float v = w * load_elem<D, BF16>(vkp, (uint64_t)rc * k + e);
#pragma unroll
        for (int g = 0; g < G; ++g) a[g] = fmaf(q_lds[c * G + g], v, a[g]);
      }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float t = group_sum<LPRK>(a[g]) * P.scale_log2;
      t = row < T ? t : -INFINITY;
      mx[g] = fmaxf(mx[g], t);
      a[g] = t;
    }
    if (ks == 0) {
#pragma unroll
      for (int g = 0; g < G; ++g) s_lds[wave][g][pass * RPK + kr] = a[g];
    }
  }
  // Token-level residual set: the wave's 128 tokens are one chunk of the
  // running counts; the logits of the set's tokens get q . sum_f w_f H_f
  // (lanes over channels, one token at a time) before the max.
  const int NF = P.bsize - 1;
  int ntr = 0;
  uint32_t tbase = 0;
  const uint8_t* hkp = nullptr;
  const uint8_t* hvp = nullptr;
  const uint32_t* tmask = nullptr;
  if (tokres) {
    const TokLayout Lt = tok_layout(mode, (uint64_t)T, D, unit_ppm(P.res_ppm, P.n_rates, P.rates_ppm, mbyte), E, E,
                                    P.bsize);
    tmask = reinterpret_cast<const uint32_t*>(seg + Lt.mask);
    tbase = reinterpret_cast<const uint32_t*>(seg + Lt.count)[wtok0 / kTokChunk];
    hkp = seg + Lt.hk;
    hvp = seg + Lt.hv;
    __syncthreads();  // the K pass's logits are in LDS
    for (int tl = 0; tl < CH; ++tl) {
      const int row = wtok0 + tl;
      if (row >= T || !((tmask[row >> 5] >> (row & 31)) & 1u)) continue;
      const uint64_t h0 = (uint64_t)(tbase + ntr) * NF * D;
      for (int g = 0; g < G; ++g) {
        float a = 0.f;
        for (int c = lane; c < D; c += 64) {
          float hsum = 0.f;
          for (int f = 0; f < NF; ++f) hsum = fmaf(P.wres[f], load_elem<D, BF16>(hkp, h0 + (uint64_t)f * D + c), hsum);
          a = fmaf(q_lds[c * G + g], hsum, a);
        }
        a = wave_sum(a) * P.scale_log2;
        if (lane == 0) s_lds[wave][g][tl] += a;
      }
      ++ntr;
    }
    __syncthreads();
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float x = -INFINITY;
      for (int tl = lane; tl < CH; tl += 64) x = fmaxf(x, s_lds[wave][g][tl]);
      mx[g] = x;
    }
  }
  float m[G];
#pragma unroll
  for (int g = 0; g < G; ++g) m[g] = wave_max(mx[g]);
  __syncthreads();

  // ------------------------------------------------------------ probabilities
  float lsum[G];
#pragma unroll
  for (int g = 0; g < G; ++g) lsum[g] = 0.f;
#pragma unroll
  for (int i = 0; i < CH / 64; ++i) {
    const int t = i * 64 + lane;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float s = s_lds[wave][g][t];
      const float p = (s == -INFINITY) ? 0.f : exp2f(s - m[g]);
      lsum[g] += p;
      s_lds[wave][g][t] = p;
      if constexpr (BF16) {
        const int ii = t / RPV, r = t % RPV;
        reinterpret_cast<uint16_t*>(&pp_lds[wave][g][0])[((ii >> 1) * RPV + r) * 2 + (ii & 1)] =
            (uint16_t)f32_to_bf16_bits(p);
      }
    }
  }
#pragma unroll
  for (int g = 0; g < G; ++g) lsum[g] = wave_sum(lsum[g]);
  __syncthreads();

  // ------------------------------------------------------------ V pass
  const int vr = lane / NP, vpc = lane % NP;
  float acc[G][CPP];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int c = 0; c < CPP; ++c) acc[g][c] = 0.f;
  if constexpr (BF16) {
    for (int ii = 0; ii < CH / RPV; ii += 2) {
      const int ra = min(wtok0 + ii * RPV + vr, T - 1);
      const int rb = min(wtok0 + (ii + 1) * RPV + vr, T - 1);
      const uint4 va = *reinterpret_cast<const uint4*>(vplane + (uint64_t)ra * RB + vpc * 16);
      const uint4 vb = *reinterpret_cast<const uint4*>(vplane + (uint64_t)rb * RB + vpc * 16);
      uint32_t pp[G];
#pragma unroll
      for (int g = 0; g < G; ++g) pp[g] = pp_lds[wave][g][(ii >> 1) * RPV + vr];
      const uint32_t* wa = reinterpret_cast<const uint32_t*>(&va);
      const uint32_t* wb = reinterpret_cast<const uint32_t*>(&vb);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint32_t lo = __builtin_amdgcn_perm(wb[w], wa[w], 0x05040100u);
        const uint32_t hi = __builtin_amdgcn_perm(wb[w], wa[w], 0x07060302u);
#pragma unroll
        for (int g = 0; g < G; ++g) {
          acc[g][2 * w] = dot2_bf16(lo, pp[g], acc[g][2 * w]);
          acc[g][2 * w + 1] = dot2_bf16(hi, pp[g], acc[g][2 * w + 1]);
        }
      }
    }
  } else {
    for (int ii = 0; ii < CH / RPV; ++ii) {
      const int tl = ii * RPV + vr;
      const int rr = min(wtok0 + tl, T - 1);
      const float4 v = *reinterpret_cast<const float4*>(vplane + (uint64_t)rr * RB + vpc * 16);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float p = s_lds[wave][g][tl];
        acc[g][0] = fmaf(p, v.x, acc[g][0]);
        acc[g][1] = fmaf(p, v.y, acc[g][1]);
        acc[g][2] = fmaf(p, v.z, acc[g][2]);
        acc[g][3] = fmaf(p, v.w, acc[g][3]);
      }
    }
  }
  if (tokres) {
    // V of the set's tokens: each lane owns distinct channels of the accumulator
    int j = 0;
    for (int tl = 0; tl < CH; ++tl) {
      const int row = wtok0 + tl;
      if (row >= T || !((tmask[row >> 5] >> (row & 31)) & 1u)) continue;
      const uint64_t h0 = (uint64_t)(tbase + j) * NF * D;
      for (int c = lane; c < D; c += 64) {
        float hsum = 0.f;
        for (int f = 0; f < NF; ++f) hsum = fmaf(P.wres[f], load_elem<D, BF16>(hvp, h0 + (uint64_t)f * D + c), hsum);
#pragma unroll
        for (int g = 0; g < G; ++g) sp_lds[wave][g][c] += s_lds[wave][g][tl] * hsum;
      }
      ++j;
    }
  }
  if (resid) {
    const int ne = CH * k;
    for (int e = lane; e < ne; e += 64) {
      const int tl = e / k, j = e - tl * k;
      const int row = wtok0 + tl;
      if (row < T) {
        float w;
        const int c = entry(ivp, (uint64_t)row * k + j, w);
        const float v = w * load_elem<D, BF16>(vvp, (uint64_t)row * k + j);
#pragma unroll
        for (int g = 0; g < G; ++g) atomicAdd(&sp_lds[wave][g][c], s_lds[wave][g][tl] * v);
      }
    }
  }
#pragma unroll
  for (int off = NP; off < 64; off <<= 1)
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int c = 0; c < CPP; ++c) acc[g][c] += __shfl_xor(acc[g][c], off, 64);
  __syncthreads();
  if (lane < NP) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int c = 0; c < CPP; ++c) mg_lds[wave][g][lane * CPP + c] = acc[g][c] + sp_lds[wave][g][lane * CPP + c];
  }
  if (lane == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      mg_lds[wave][g][D] = m[g];
      mg_lds[wave][g][D + 1] = lsum[g];
    }
  }
  __syncthreads();

  // ------------------------------------------------------------ merge waves
  float* rec = P.ws + ((uint64_t)sh * P.n_chunks_total + slot) * G * S::RS;
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
        const float f = (mw == -INFINITY) ? 0.f : exp2f(mw - M);
        o = fmaf(f, mg_lds[w][g][c], o);
      }
    }
    rec[g * S::RS + c] = o;
  }
}

template <int D, bool BF16, int G>
static hipError_t launch_decode_t(const DecodeParams& P, hipStream_t s) {
  static_assert(!BF16, "bf16 caches use decode_stream_kernel");
  const dim3 grid((unsigned)P.batch * P.hkv * P.n_chunks_total);
  if (grid.x > 0) hipLaunchKernelGGL((decode_splitk_kernel<D, BF16, G>), grid, dim3(256), 0, s, P);
  return hipGetLastError();
}

template <int D, bool BF16>
static hipError_t launch_decode_d(const DecodeParams& P, hipStream_t s) {
  switch (P.hq / P.hkv) {
    case 1: return launch_decode_t<D, BF16, 1>(P, s);
    case 2: return launch_decode_t<D, BF16, 2>(P, s);
    case 4: return launch_decode_t<D, BF16, 4>(P, s);
    default: return launch_decode_t<D, BF16, 8>(P, s);
  }
}

hipError_t launch_decode(const DecodeParams& P, hipStream_t s) {
  if (P.bf16) return launch_decode_stream(P, s);
  return P.d == 128 ? launch_decode_d<128, false>(P, s) : launch_decode_d<64, false>(P, s);
}

}  // namespace fdkv
