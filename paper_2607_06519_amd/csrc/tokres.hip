// Token-level residual set (Section 3, the paragraph after Eq. 2): a
// residual head keeps every high-frequency depth coefficient of the r*T
// tokens whose removal would change a probe logit the most,
//   s_t = max over probe rows q of |q . (K_t - K^S_t)|,
// and stores the shared reconstruction for all others (Eq. 3 with the set S
// of those tokens).
//
// Kernels:
//  * token_score - the probe's logits against the deviations K - K^S of
//    every layer of the block, with v_mfma_f32_32x32x16_bf16: probe rows
//    (staged in LDS, shared by the workgroup's eight waves) times the
//    deviations of 64 tokens per wave (built in registers from the inputs:
//    fp32 arithmetic rounded to bf16 for the MFMA, so a score lies within
//    (2^-9 + 2^-16) max_q sum_c |q_c| |dev_c| of its exact value).  Per
//    token: the largest |logit| (the score) and the sum of squares (its
//    share of Eq. 2).  fp32 queries go in as two bf16 halves.
//  * token_select - one workgroup per unit: the n-th largest score by a
//    4-pass radix select over the score bits (scores are >= 0, so their bits
//    order like the values), then every score above it and the first scores
//    equal to it in token order.  Probe: E_S and E_R from the sums of
//    squares.  Compress: the token mask and the running counts.
//  * token_rows - one workgroup per 128-token chunk of a residual unit: the
//    high-frequency coefficients of the chunk's selected tokens (pairs: the
//    half difference; fours: Z_1..Z_3 of the DCT-II(4) butterfly), written
//    at their running count.
#include "fdkv_common.h"
#include "fdkv_kernels.h"
#include "fp8.h"

namespace fdkv {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
constexpr int kRsrcWord3 = 0x00020000;
constexpr uint32_t kOobOff = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint64_t bytes) {
  const uint32_t n = bytes > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, kRsrcWord3);
}

__device__ __forceinline__ uint4 load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

__device__ __forceinline__ uint32_t w4(const uint4& v, int i) { return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w; }

// 8 consecutive channels of a row as fp32: bf16 rows take one 16-byte piece,
// fp32 rows two.
template <bool BF16>
__device__ __forceinline__ void load8(__amdgpu_buffer_rsrc_t r, uint32_t off, bool ok, float (&x)[8]) {
  if constexpr (BF16) {
    const uint4 v = load16(r, ok ? off : kOobOff);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = bf16_lo(w4(v, i));
      x[2 * i + 1] = bf16_hi(w4(v, i));
    }
  } else {
    const uint4 a = load16(r, ok ? off : kOobOff), b = load16(r, ok ? off + 16 : kOobOff);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[i] = as_f32(w4(a, i));
      x[4 + i] = as_f32(w4(b, i));
    }
  }
}

// The deviations K - K^S of layer l of a block, 8 channels, in fp32 and
// without fused multiply-adds (the score's precision; rounded to bf16 by the
// caller).  Pairs: (x0 - x1) / 2 for layer 0 and its negation for layer 1;
// fours: x_l - ((x0 + x3) + (x1 + x2)) / 4.
template <int NB>
__device__ __forceinline__ float deviation(const float (&x)[NB][8], int l, int c) {
#pragma clang fp contract(off)
  if constexpr (NB == 2) {
    const float dd = (x[0][c] - x[1][c]) * 0.5f;
    return l == 0 ? dd : -dd;
  } else {
    const float m = ((x[0][c] + x[3][c]) + (x[1][c] + x[2][c])) * 0.25f;
    return x[l][c] - m;
  }
}

__device__ __forceinline__ bf16x8_t pack8(const float (&v)[8]) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = pack_bf16x2(v[2 * i], v[2 * i + 1]);
  return __builtin_bit_cast(bf16x8_t, make_uint4(w[0], w[1], w[2], w[3]));
}

}  // namespace

// ---------------------------------------------------------------- scores
// Eight waves (512 tokens) per workgroup share each round of probe rows in
// LDS: half the probe-row traffic of four waves, 2.35 -> 2.25 ms on the 8B
// token-set probe (sixteen waves, or 64 rows a round, lose occupancy).
constexpr int kScoreThreads = 512;

template <int D, bool BF16, int NB>
__global__ __launch_bounds__(kScoreThreads) void token_score_kernel(TokenParams P) {
  constexpr int TH = kScoreThreads;
  constexpr int E = BF16 ? 2 : 4;
  constexpr int KS = D / 16;                 // k-steps of the 32x32x16 MFMA
  constexpr int NPQ = D / 8;                 // 8-channel pieces of a probe row
  constexpr int LDR = D + 8;                 // LDS row stride (bf16 elements): 16-byte pad
  constexpr int NH = BF16 ? 1 : 2;           // bf16 halves of a query (fp32 queries: hi + lo)
  constexpr int NL = NB == 2 ? 1 : NB;       // deviation passes (a pair's two layers share one up to sign)
  __shared__ __attribute__((aligned(16))) uint16_t qs[NH][32 * LDR];

  const int bi = blockIdx.y / P.hkv, head = blockIdx.y % P.hkv;
  const int first = P.bl.first[bi];
  const int unit = P.bl.block[bi] * P.hkv + head;
  const int T = P.seq_len, G = P.hq / P.hkv, GP = G * P.n_probe;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const uint64_t RB = (uint64_t)D * E;
  const uint64_t plane = (uint64_t)T * RB;
  __amdgpu_buffer_rsrc_t kr[NB];
#pragma unroll
  for (int n = 0; n < NB; ++n)
    kr[n] = make_rsrc(static_cast<const uint8_t*>(P.k[first + n]) + (uint64_t)head * plane, plane);
  const uint64_t qspan = (uint64_t)GP * RB;  // one layer's probe rows of this KV head

  const int tl = lane & 31, kh = lane >> 5;
  const int tok_w = blockIdx.x * TH + wave * 64;   // the wave's 64 tokens: two sets of 32
  float mx[2] = {0.f, 0.f}, ss[2] = {0.f, 0.f};

  for (int pass = 0; pass < NL; ++pass) {
    // B operands: the deviation rows of the wave's tokens for this pass
    bf16x8_t bop[2][KS];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const int t = tok_w + st * 32 + tl;
      const bool ok = t < T;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const uint32_t off = (uint32_t)t * (uint32_t)RB + (uint32_t)((2 * ks + kh) * 8 * E);
        float x[NB][8];
#pragma unroll
        for (int n = 0; n < NB; ++n) load8<BF16>(kr[n], off, ok, x[n]);
        float dv[8];
#pragma unroll
        for (int c = 0; c < 8; ++c) dv[c] = deviation<NB>(x, pass, c);
        bop[st][ks] = pack8(dv);
      }
    }
    // probe rows: the pass's layer(s), 32 rows at a time through LDS
    const int nlay = NB == 2 ? 2 : 1;
    for (int ly = 0; ly < nlay; ++ly) {
      const int layer = first + (NB == 2 ? ly : pass);
      const auto qr = make_rsrc(static_cast<const uint8_t*>(P.qp[layer]) + (uint64_t)head * qspan, qspan);
      // 32 probe rows per round; the next round's rows are loaded into
      // registers while this round's MFMAs run
      constexpr int PER = (32 * NPQ + TH - 1) / TH;  // 8-channel pieces per thread and round
      float qn[PER][8];
      auto fetch = [&](int r0) {
#pragma unroll
        for (int j = 0; j < PER; ++j) {
          const int i = tid + TH * j, row = i / NPQ, pc = i % NPQ;
          load8<BF16>(qr, (uint32_t)((r0 + row) * RB + pc * 8 * E), i < 32 * NPQ && r0 + row < GP, qn[j]);
        }
      };
      fetch(0);
      for (int r0 = 0; r0 < GP; r0 += 32) {
        __syncthreads();  // the previous round's rows are read
#pragma unroll
        for (int j = 0; j < PER; ++j) {
          const int i = tid + TH * j, row = i / NPQ, pc = i % NPQ;
          if (i >= 32 * NPQ) continue;
          const float* q = qn[j];
          uint32_t hi[4], lo[4];
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            hi[jj] = pack_bf16x2(q[2 * jj], q[2 * jj + 1]);
            if constexpr (NH == 2)
              lo[jj] = pack_bf16x2(q[2 * jj] - bf16_lo(hi[jj]), q[2 * jj + 1] - bf16_hi(hi[jj]));
          }
          *reinterpret_cast<uint4*>(&qs[0][row * LDR + pc * 8]) = make_uint4(hi[0], hi[1], hi[2], hi[3]);
          if constexpr (NH == 2)
            *reinterpret_cast<uint4*>(&qs[NH - 1][row * LDR + pc * 8]) = make_uint4(lo[0], lo[1], lo[2], lo[3]);
        }
        __syncthreads();
        if (r0 + 32 < GP) fetch(r0 + 32);
        f32x16_t acc[2];
#pragma unroll
        for (int st = 0; st < 2; ++st)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[st][r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
          for (int h = 0; h < NH; ++h) {
            const bf16x8_t aop = *reinterpret_cast<const bf16x8_t*>(&qs[h][tl * LDR + ks * 16 + kh * 8]);
#pragma unroll
            for (int st = 0; st < 2; ++st)
              acc[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(aop, bop[st][ks], acc[st], 0, 0, 0);
          }
        }
        // lane holds 16 rows of its token (column tl); rows past GP are zero rows
#pragma unroll
        for (int st = 0; st < 2; ++st)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float v = acc[st][r];
            mx[st] = fmaxf(mx[st], fabsf(v));
            ss[st] = fmaf(v, v, ss[st]);
          }
      }
    }
  }
  // lanes l and l + 32 saw the other 16 rows of each block for the same token
#pragma unroll
  for (int st = 0; st < 2; ++st) {
    mx[st] = fmaxf(mx[st], __shfl_xor(mx[st], 32, 64));
    ss[st] += __shfl_xor(ss[st], 32, 64);
  }
  if (kh == 0) {
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const int t = tok_w + st * 32 + tl;
      if (t < T) {
        P.scores[(uint64_t)unit * T + t] = mx[st];
        if (P.sumsq) P.sumsq[(uint64_t)unit * T + t] = ss[st];
      }
    }
  }
}

// ---------------------------------------------------------------- selection
namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelBatch = 16;   // keys per thread and batch of a radix pass
constexpr int kSelGroups = 8;   // groups of 64 tokens per batch of a wave's walk

}  // namespace

// Probe (P.modes null): for every candidate fraction of the cache (res_ppm,
// or each of the n_rates routed ones) the set's share of the loss, written as
// errors [unit][1 + J] = E_S, E_R(r_0), ..., E_R(r_{J-1}).  Compress: the set of
// the unit's own fraction (its mode byte), as the token mask and the running
// counts.
__global__ __launch_bounds__(kSelThreads) void token_select_kernel(TokenParams P) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t pick[2];
  __shared__ uint32_t run_eq[kSelThreads / 64], run_gt[kSelThreads / 64];
  __shared__ double red[kSelThreads / 64][2];
  const int bi = blockIdx.x / P.hkv, head = blockIdx.x % P.hkv;
  const int unit = P.bl.block[bi] * P.hkv + head;
  if (P.modes && mode_of(P.modes[unit]) != kResidual) return;
  const int T = P.seq_len, tid = threadIdx.x;
  const uint32_t* key = reinterpret_cast<const uint32_t*>(P.scores + (uint64_t)unit * T);
  const int J = P.modes ? 1 : (P.n_rates ? P.n_rates : 1);
  for (int jr = 0; jr < J; ++jr) {
  const int ppm = P.modes ? unit_ppm(P.res_ppm, P.n_rates, P.rates_ppm, P.modes[unit])
                          : (P.n_rates ? P.rates_ppm[jr] : P.res_ppm);
  const uint32_t n = (uint32_t)min<uint64_t>(residual_token_count((uint64_t)T, ppm), (uint64_t)T);

  // 1. tau = the n-th largest key, need = how many keys equal to tau are taken
  uint32_t prefix = 0, pmask = 0, need = n;
  for (int shift = 24; shift >= 0 && n > 0; shift -= 8) {
    if (tid < 256) hist[tid] = 0;
    __syncthreads();
    // kSelBatch keys per thread in flight, then their counts
    for (int t0 = tid; t0 < T; t0 += kSelBatch * kSelThreads) {
      uint32_t kb[kSelBatch];
#pragma unroll
      for (int j = 0; j < kSelBatch; ++j) {
        const int t = t0 + j * kSelThreads;
        kb[j] = t < T ? key[t] : 0u;
      }
#pragma unroll
      for (int j = 0; j < kSelBatch; ++j)
        if (t0 + j * kSelThreads < T && (kb[j] & pmask) == prefix) atomicAdd(&hist[(kb[j] >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < 64) {
      // the digit: the highest bin b whose count of keys in bins >= b
      // reaches need (the suffix counts fall with b, so b + 1 is how many
      // bins reach it); lane l holds bins 4l .. 4l + 3
      const uint32_t h0 = hist[4 * tid], h1 = hist[4 * tid + 1], h2 = hist[4 * tid + 2], h3 = hist[4 * tid + 3];
      const uint32_t mine = h0 + h1 + h2 + h3;
      uint32_t incl = mine;  // keys in this lane's bins and above
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_down(incl, o, 64);
        if (tid + o < 64) incl += y;
      }
      const uint32_t s3 = incl - mine + h3, s2 = s3 + h2, s1 = s2 + h1, s0 = s1 + h0;
      uint32_t c = (s0 >= need) + (s1 >= need) + (s2 >= need) + (s3 >= need);
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) c += __shfl_xor(c, o, 64);
      const uint32_t bstar = c > 0 ? c - 1 : 0;
      if ((uint32_t)tid == bstar >> 2) {
        const uint32_t j = bstar & 3u;
        const uint32_t sj = j == 0 ? s0 : j == 1 ? s1 : j == 2 ? s2 : s3;
        const uint32_t hj = j == 0 ? h0 : j == 1 ? h1 : j == 2 ? h2 : h3;
        pick[0] = bstar;
        pick[1] = need - (sj - hj);  // need less the keys in the bins above b
      }
    }
    __syncthreads();
    prefix |= pick[0] << shift;
    pmask |= 255u << shift;
    need = pick[1];
    __syncthreads();
  }
  const uint32_t tau = prefix;

  // 2. each wave takes a contiguous run of 128-token chunks and walks it 64
  //    tokens at a time (coalesced loads, ballots): a first walk counts the
  //    run's keys above and equal to tau, the waves' counts in order give
  //    each run the equal keys and the selected tokens before it, and a
  //    second walk ranks the equal keys in token order and emits the set
  const int lane = tid & 63, wave = tid >> 6;
  constexpr int kW = kSelThreads / 64;
  const int words = (T + 31) / 32, chunks = (T + kTokChunk - 1) / kTokChunk;
  const int cpw = (chunks + kW - 1) / kW;                     // chunks per wave
  const int c0 = min(wave * cpw, chunks), c1 = min(c0 + cpw, chunks);
  const int t0 = c0 * kTokChunk, t1 = min(c1 * kTokChunk, T);
  uint32_t n_eq = 0, n_gt = 0;
  if (n > 0)
    for (int g0 = t0; g0 < t1; g0 += kSelGroups * 64) {  // kSelGroups groups of 64 tokens in flight
      uint32_t kb[kSelGroups];
#pragma unroll
      for (int j = 0; j < kSelGroups; ++j) {
        const int t = g0 + 64 * j + lane;
        kb[j] = t < t1 ? key[t] : 0u;
      }
#pragma unroll
      for (int j = 0; j < kSelGroups; ++j) {
        const bool ok = g0 + 64 * j + lane < t1;
        n_eq += (uint32_t)__popcll(__ballot(ok && kb[j] == tau));
        n_gt += (uint32_t)__popcll(__ballot(ok && kb[j] > tau));
      }
    }
  if (lane == 0) {
    run_eq[wave] = n_eq;
    run_gt[wave] = n_gt;
  }
  __syncthreads();
  // equal keys and selected tokens before this run, and the set's size:
  // a run takes its keys above tau and the equal ones still needed
  uint32_t eq_acc = 0, rank = 0, sel_run = 0, sel_total = 0;
  for (int w = 0; w < kW; ++w) {
    if (w == wave) {
      rank = eq_acc;
      sel_run = sel_total;
    }
    sel_total += run_gt[w] + (need > eq_acc ? min(run_eq[w], need - eq_acc) : 0u);
    eq_acc += run_eq[w];
  }
  double sum_all = 0.0, sum_kept = 0.0;
  uint32_t* mask_out = nullptr;
  uint32_t* count_out = nullptr;
  if (P.modes) {
    uint8_t* seg = P.cache + P.seg_off[unit];
    const TokLayout L = tok_layout(kResidual, (uint64_t)T, P.d, ppm, P.bf16 ? 2 : 4,
                                   P.bf16 ? (P.coef8 ? 1 : 2) : 4, P.bsize);
    mask_out = reinterpret_cast<uint32_t*>(seg + L.mask);
    count_out = reinterpret_cast<uint32_t*>(seg + L.count);
  }
  const uint64_t below = (1ull << lane) - 1ull;
  for (int g0 = t0; g0 < t1; g0 += kSelGroups * 64) {
    // kSelGroups groups of 64 tokens: keys and losses in flight, then in token order
    uint32_t kb[kSelGroups];
    float eb[kSelGroups];
#pragma unroll
    for (int j = 0; j < kSelGroups; ++j) {
      const int t = g0 + 64 * j + lane;
      kb[j] = t < t1 ? key[t] : 0u;
      eb[j] = (P.sumsq && t < t1) ? P.sumsq[(uint64_t)unit * T + t] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < kSelGroups; ++j) {
      const int g = g0 + 64 * j;
      if (g >= t1) break;
      const int t = g + lane;
      const bool ok = t < t1;
      const uint32_t k = kb[j];
      const bool eq = ok && n > 0 && k == tau;
      const uint64_t beq = __ballot(eq);
      const uint32_t r = rank + (uint32_t)__popcll(beq & below);
      const bool sel = ok && n > 0 && (k > tau || (eq && r < need));
      rank += (uint32_t)__popcll(beq);
      const uint64_t bsel = __ballot(sel);
      // 3. compress: the token mask, and the running count before every chunk
      if (mask_out) {
        if (lane == 0) mask_out[g >> 5] = (uint32_t)bsel;
        if (lane == 32 && (g >> 5) + 1 < words) mask_out[(g >> 5) + 1] = (uint32_t)(bsel >> 32);
      }
      if (count_out && lane == 0 && (g & (kTokChunk - 1)) == 0) count_out[g / kTokChunk] = sel_run;
      sel_run += (uint32_t)__popcll(bsel);
      if (P.sumsq && ok) {
        const double e = (double)eb[j];
        sum_all += e;
        sum_kept += sel ? e : 0.0;
      }
    }
  }
  if (count_out && tid == 0) count_out[chunks] = sel_total;
  //    probe: the losses
  if (P.sumsq) {
    // fixed-order reduction: waves by shuffles, then wave 0 over the 16 partials
    const int lane = tid & 63, wave = tid >> 6;
    double a = sum_all, b = sum_all - sum_kept;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      a += __shfl_xor(a, o, 64);
      b += __shfl_xor(b, o, 64);
    }
    if (lane == 0) {
      red[wave][0] = a;
      red[wave][1] = b;
    }
    __syncthreads();
    if (tid < 2 && (tid == 1 || jr == 0)) {
      double s = 0.0;
      for (int w = 0; w < kSelThreads / 64; ++w) s += red[w][tid];
      const double norm = (double)P.bsize * (P.hq / P.hkv) * (double)P.n_probe * (double)P.d;
      P.errors[(uint64_t)unit * (1 + J) + (tid ? 1 + jr : 0)] = (float)(s / norm);
    }
    __syncthreads();  // red, hist and pick are reused by the next fraction
  }
  }  // fractions
}

// ---------------------------------------------------------------- rows
template <int D, bool BF16, int NB>
__global__ __launch_bounds__(256) void token_rows_kernel(TokenParams P) {
  constexpr int E = BF16 ? 2 : 4;
  constexpr int NPc = D / 8;               // 8-channel pieces of a row
  constexpr int NF = NB - 1;               // high-frequency rows per token
  __shared__ int list[kTokChunk];
  const int chunk = blockIdx.x;
  const int bi = blockIdx.y / P.hkv, head = blockIdx.y % P.hkv;
  const int first = P.bl.first[bi];
  const int unit = P.bl.block[bi] * P.hkv + head;
  if (mode_of(P.modes[unit]) != kResidual) return;
  const int T = P.seq_len, tid = threadIdx.x;
  const bool c8 = BF16 && P.coef8;
  const int CE = c8 ? 1 : E;
  uint8_t* seg = P.cache + P.seg_off[unit];
  const TokLayout L = tok_layout(kResidual, (uint64_t)T, D, unit_ppm(P.res_ppm, P.n_rates, P.rates_ppm, P.modes[unit]),
                                 E, CE, NB);
  const uint32_t* mask = reinterpret_cast<const uint32_t*>(seg + L.mask);
  const uint32_t base = reinterpret_cast<const uint32_t*>(seg + L.count)[chunk];
  const int t0 = chunk * kTokChunk;

  // the chunk's selected tokens, in order: threads 0..127 own one token each
  // (waves 0 and 1); every thread takes part in the ballot and the barrier
  __shared__ uint32_t wave_n[2];
  const int lane = tid & 63, wave = tid >> 6;
  bool sel = false;
  if (tid < kTokChunk) {
    const int t = t0 + tid;
    sel = t < T && ((mask[t >> 5] >> (t & 31)) & 1u);
  }
  const uint64_t bal = __ballot(sel);
  if (lane == 0 && wave < 2) wave_n[wave] = (uint32_t)__builtin_popcountll(bal);
  __syncthreads();
  if (sel) {
    const uint32_t below = (uint32_t)__builtin_popcountll(bal & ((1ull << lane) - 1ull));
    list[below + (wave == 1 ? wave_n[0] : 0u)] = tid;
  }
  const int nsel = (int)(wave_n[0] + wave_n[1]);
  __syncthreads();

  const uint64_t RB = (uint64_t)D * E, plane = (uint64_t)T * RB, hoff = (uint64_t)head * plane;
  const uint64_t rowc = (uint64_t)NF * D * CE;      // bytes of one token's rows
  for (int it = tid; it < nsel * NPc * 2; it += 256) {
    const int j = it / (NPc * 2), rem = it % (NPc * 2), tensor = rem / NPc, pc = rem % NPc;
    const int t = t0 + list[j];
    const void* const* src = tensor ? P.v : P.k;
    float x[NB][8];
#pragma unroll
    for (int n = 0; n < NB; ++n) {
      const uint8_t* p = static_cast<const uint8_t*>(src[first + n]) + hoff + (uint64_t)t * RB + (uint64_t)pc * 8 * E;
#pragma unroll
      for (int c = 0; c < 8; ++c)
        x[n][c] = BF16 ? bf16_to_f32(reinterpret_cast<const uint16_t*>(p)[c]) : reinterpret_cast<const float*>(p)[c];
    }
    float h[NF][8];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      if constexpr (NB == 2) {
        h[0][c] = (x[0][c] - x[1][c]) * 0.5f;
      } else {
        dct4_high(x[0][c], x[1][c], x[2][c], x[3][c], h[0][c], h[1][c], h[2][c]);
      }
    }
    uint8_t* dst = seg + (tensor ? L.hv : L.hk) + (uint64_t)(base + j) * rowc;
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      uint8_t* o = dst + ((uint64_t)f * D + pc * 8) * CE;
      if (c8) {
        *reinterpret_cast<uint2*>(o) = make_uint2(e4m3_quad(h[f][0], h[f][1], h[f][2], h[f][3]),
                                                  e4m3_quad(h[f][4], h[f][5], h[f][6], h[f][7]));
      } else if constexpr (BF16) {
        *reinterpret_cast<uint4*>(o) = make_uint4(pack_bf16x2(h[f][0], h[f][1]), pack_bf16x2(h[f][2], h[f][3]),
                                                  pack_bf16x2(h[f][4], h[f][5]), pack_bf16x2(h[f][6], h[f][7]));
      } else {
        *reinterpret_cast<float4*>(o) = make_float4(h[f][0], h[f][1], h[f][2], h[f][3]);
        *reinterpret_cast<float4*>(o + 16) = make_float4(h[f][4], h[f][5], h[f][6], h[f][7]);
      }
    }
  }
}

// ---------------------------------------------------------------- launchers
template <int D, bool BF16, int NB>
static hipError_t launch_scores_t(const TokenParams& P, hipStream_t s) {
  const dim3 grid((P.seq_len + kScoreThreads - 1) / kScoreThreads, P.bl.n * P.hkv);
  hipLaunchKernelGGL((token_score_kernel<D, BF16, NB>), grid, dim3(kScoreThreads), 0, s, P);
  return hipGetLastError();
}

template <int D, bool BF16>
static hipError_t launch_scores_d(const TokenParams& P, hipStream_t s) {
  return P.bsize == 4 ? launch_scores_t<D, BF16, 4>(P, s) : launch_scores_t<D, BF16, 2>(P, s);
}

hipError_t launch_token_scores(const TokenParams& P, hipStream_t s) {
  if (P.bl.n == 0 || P.seq_len == 0) return hipSuccess;
  if (P.d == 128) return P.bf16 ? launch_scores_d<128, true>(P, s) : launch_scores_d<128, false>(P, s);
  return P.bf16 ? launch_scores_d<64, true>(P, s) : launch_scores_d<64, false>(P, s);
}

hipError_t launch_token_select(const TokenParams& P, hipStream_t s) {
  if (P.bl.n == 0 || P.seq_len == 0) return hipSuccess;
  hipLaunchKernelGGL(token_select_kernel, dim3(P.bl.n * P.hkv), dim3(kSelThreads), 0, s, P);
  return hipGetLastError();
}

template <int D, bool BF16, int NB>
static hipError_t launch_rows_t(const TokenParams& P, hipStream_t s) {
  const dim3 grid((P.seq_len + kTokChunk - 1) / kTokChunk, P.bl.n * P.hkv);
  hipLaunchKernelGGL((token_rows_kernel<D, BF16, NB>), grid, dim3(256), 0, s, P);
  return hipGetLastError();
}

template <int D, bool BF16>
static hipError_t launch_rows_d(const TokenParams& P, hipStream_t s) {
  return P.bsize == 4 ? launch_rows_t<D, BF16, 4>(P, s) : launch_rows_t<D, BF16, 2>(P, s);
}

hipError_t launch_token_rows(const TokenParams& P, hipStream_t s) {
  if (P.bl.n == 0 || P.seq_len == 0) return hipSuccess;
  if (P.d == 128) return P.bf16 ? launch_rows_d<128, true>(P, s) : launch_rows_d<128, false>(P, s);
  return P.bf16 ? launch_rows_d<64, true>(P, s) : launch_rows_d<64, false>(P, s);
}

}  // namespace fdkv
