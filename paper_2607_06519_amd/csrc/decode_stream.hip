// Streaming split-K decode over a bf16 compressed cache (Section 3: the
// reconstruction of Eq. 3 fused into the attention).
//
// One workgroup = 4 waves = 512 tokens of one (sequence, KV head); a wave
// walks 128 of them in 8-row tiles (d = 128; 16 rows at d = 64) with an
// online softmax, keeping the next tiles' loads in flight while it computes
// the current one.  The waves take the workgroup's tiles in turn (tile t of
// wave w: tile 4t + w), so at any time they read one short run of each
// plane; the rows of a token-level set are taken afterwards by the wave
// whose 128 consecutive tokens (one chunk of the running counts) hold them.
//
// One lane layout serves the K pass, the softmax and the V pass: NP = d/8
// lanes per token row, each holding one 16-byte piece (8 channels), so one
// load instruction covers RPL = 64/NP consecutive rows and a lane owns
// NL = TILE/RPL rows of a tile (two).  The NP lanes of a row form a DPP row (d = 128)
// or half row (d = 64).
//  K   - bf16 dot2 of the lane's piece with its piece of every query (held in
//        registers); residual heads add the lane's residual entry
//        w * q[c] * value (B = 2: c the channel, w = +-1 for the stored half
//        difference; B = 4: code 4c + j, w = F_4[j][p] for layer p of the
//        block); a DPP reduce-scatter over the row's lanes then leaves each
//        lane one full (row, head) logit (2G <= NP: d = 128, or d = 64 with
//        G <= 4; d = 64 with G = 8 sums every logit on every lane instead);
//  max - a running reference max per head, equal on the lanes of that head,
//        that moves (the head's max over the wave, rescale by
//        exp2(m_old - m_new)) only when a logit exceeds it by more than 2^8;
//        scale, mask, exp2 and running sum run once per logit;
//  V   - each lane's probability goes back to the row as a bf16 pair (the
//        same head's other row) and an all-gather over the heads, so nothing
//        goes through LDS; the lane's two rows share one dot2 that
//        multiplies two tokens' values by their probabilities; residual heads add
//        w * p * value into LDS accumulators, one copy per row of a load
//        (a row's entries sit on distinct channels for B = 2, so a plain
//        read-add-write is safe; for B = 4 up to three frequencies of one
//        channel sit in adjacent lanes, since codes 4c + j are stored
//        ascending: a DPP pass hands each run's sum to its first lane and
//        only that lane writes, which keeps the adds plain as well -- LDS
//        float atomics tripled the layer time).
// The 4 waves merge in LDS and write one (acc, m, l) record per workgroup;
// decode_merge combines the records.  HBM bound: no MFMA.
#include "fdkv_common.h"
#include "fdkv_kernels.h"

#include <type_traits>

namespace fdkv {

namespace {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
constexpr int kRsrcDword3 = 0x00020000;  // raw buffer, 32-bit data format (gfx9 family)
constexpr float kSlack = 8.f;            // log2 headroom of the running reference max
constexpr uint32_t kOob = 0x80000000u;   // buffer offset past every plane (planes are < 2^31 bytes): loads read 0

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

// The K and V tile loads and the residual entries: every byte of a plane is
// read once per decode step, so they carry the non-temporal cache hint
// (cache policy NT).
constexpr int kNonTemporal = 2;
__device__ __forceinline__ uint4 ld128_stream(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kNonTemporal);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

__device__ __forceinline__ uint32_t word(const uint4& v, int w) {
  return w == 0 ? v.x : w == 1 ? v.y : w == 2 ? v.z : v.w;
}

typedef __bf16 bf16x2v_t __attribute__((ext_vector_type(2)));

// Two FP8 E4M3 codes (bytes 0-1 or 2-3 of w) as a bf16 pair; exact, since
// every E4M3 value is a bf16 value.
template <bool HI>
__device__ __forceinline__ uint32_t e4m3x2_bf16(uint32_t w) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, HI));
}

// A piece of 8 FP8 channels (raw in .x, .y) as the 8 bf16 channels of a
// bf16 piece.
__device__ __forceinline__ uint4 widen_e4m3(const uint4& raw) {
  return make_uint4(e4m3x2_bf16<false>(raw.x), e4m3x2_bf16<true>(raw.x), e4m3x2_bf16<false>(raw.y),
                    e4m3x2_bf16<true>(raw.y));
}

// Runs of equal channels among the residual V entries of one row (blocks of
// four: codes 4c + j ascending, so a channel's frequencies are adjacent
// entries, at most three).  Lane pc holds entry e with channel c and
// contribution x; entries e - 1, e + 1, e + 2 sit in lanes pc - 1, pc + 1,
// pc + 2 of the same group of NP lanes when they exist (ok1 / ok2 say whether
// e + 1 / e + 2 exist).  Returns the run's sum on the run's first lane.
template <int NP>
__device__ __forceinline__ float run_sum(int c, float x, int pc, bool valid, bool ok1, bool ok2, bool& first) {
  constexpr int kRowShr1 = 0x111, kRowShl1 = 0x101, kRowShl2 = 0x102;
  const int cl = __builtin_amdgcn_update_dpp(-1, c, kRowShr1, 0xF, 0xF, false);
  const int c1 = __builtin_amdgcn_update_dpp(-1, c, kRowShl1, 0xF, 0xF, false);
  const int c2 = __builtin_amdgcn_update_dpp(-1, c, kRowShl2, 0xF, 0xF, false);
  const float x1 = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), kRowShl1, 0xF, 0xF, false));
  const float x2 = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), kRowShl2, 0xF, 0xF, false));
  first = valid && (pc == 0 || cl != c);
  const bool n1 = ok1 && pc + 1 < NP && c1 == c;
  const bool n2 = n1 && ok2 && pc + 2 < NP && c2 == c;
  return x + (n1 ? x1 : 0.f) + (n2 ? x2 : 0.f);
}

// Lane exchange across bit B of a row's lane index (rows of 8 or 16 lanes).
// Bits 3 and 2 use the mirrors, which also flip the lower bits: that still
// pairs each lane with one of the other half, and once the lower bits hold
// equal values (duplicates, or lists already gathered) it is the plain swap.
template <int B>
__device__ __forceinline__ uint32_t swap_bit(uint32_t x) {
  constexpr int kCtrl = B == 3 ? kDppRowMirror : B == 2 ? kDppRowHalfMirror : B == 1 ? kDppQuadXor2 : kDppQuadXor1;
  // every source lane lies in the row: bound_ctrl needs no old value
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, kCtrl, 0xF, 0xF, true);
}
template <int B>
__device__ __forceinline__ float swap_bit(float x) {
  return __uint_as_float(swap_bit<B>(__float_as_uint(x)));
}

// The lane NP/2 further along a row of NP lanes (the lane holding the same
// head for the other row of a load): row_ror:8 for 16 lanes; for 8 lanes,
// row_shl:4 into banks 0 and 2 and row_shr:4 into banks 1 and 3.
template <int NP>
__device__ __forceinline__ float swap_half(float x) {
  if constexpr (NP == 16) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x128, 0xF, 0xF, true));
  } else {
    static_assert(NP == 8, "row width");
    int y = __builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x104, 0xF, 0x5, false);
    y = __builtin_amdgcn_update_dpp(y, __float_as_int(x), 0x114, 0xF, 0xA, false);
    return __int_as_float(y);
  }
}

// One reduce-scatter stage across lane bit B: the lanes with the bit clear
// keep the list's lower half and add their partner's copy of it, the others
// the upper half.
template <int B, int H, int V>
__device__ __forceinline__ void scatter_stage(float (&a)[V], int lane) {
  const bool up = (lane >> B) & 1;
#pragma unroll
  for (int t = 0; t < H; ++t) {
    const float keep = up ? a[t + H] : a[t], send = up ? a[t] : a[t + H];
    a[t] = keep + swap_bit<B>(send);
  }
}

// Sum of V values over the 2^NPB lanes of a row, one sum per lane: the
// stages on the top log2(V) lane bits split the list (lane bits b, from the
// top, choose the half), butterflies on the lower bits finish the sums, so
// the lane holds value number (lane % 2^NPB) >> (NPB - log2 V).
template <int NPB, int V>
__device__ __forceinline__ float row_reduce_scatter(float (&a)[V], int lane) {
  constexpr int RB = V == 16 ? 4 : V == 8 ? 3 : V == 4 ? 2 : 1;
  static_assert((1 << RB) == V && RB <= NPB, "one value per lane at most");
  scatter_stage<NPB - 1, V / 2>(a, lane);
  if constexpr (RB >= 2) scatter_stage<NPB - 2, V / 4>(a, lane);
  if constexpr (RB >= 3) scatter_stage<NPB - 3, V / 8>(a, lane);
  if constexpr (RB >= 4) scatter_stage<NPB - 4, V / 16>(a, lane);
  if constexpr (NPB - RB - 1 >= 2) a[0] += swap_bit<2>(a[0]);
  if constexpr (NPB - RB - 1 >= 1) a[0] += swap_bit<1>(a[0]);
  if constexpr (NPB - RB - 1 >= 0) a[0] += swap_bit<0>(a[0]);
  return a[0];
}

// All-gather stage across lane bit B: the list of N values doubles, the
// values of lanes with the bit clear first.
template <int B, int N, int G>
__device__ __forceinline__ void gather_stage(uint32_t (&y)[G], int lane) {
  const bool up = (lane >> B) & 1;
  uint32_t o[N];
#pragma unroll
  for (int t = 0; t < N; ++t) o[t] = swap_bit<B>(y[t]);
#pragma unroll
  for (int t = 0; t < N; ++t) {
    const uint32_t mine = y[t];
    y[t] = up ? o[t] : mine;
    y[t + N] = up ? mine : o[t];
  }
}

// Every lane of a row gets the G values x of head g = (lane >> SH) % G (lanes
// that differ only below bit SH hold equal values).
template <int SH, int G>
__device__ __forceinline__ void row_gather(uint32_t x, uint32_t (&y)[G], int lane) {
  y[0] = x;
  if constexpr (G >= 2) gather_stage<SH, 1>(y, lane);
  if constexpr (G >= 4) gather_stage<SH + 1, 2>(y, lane);
  if constexpr (G >= 8) gather_stage<SH + 2, 4>(y, lane);
}

template <int D, int G>
struct SS {
  static constexpr int NP = D / 8;                 // lanes per row, one 16-byte piece each
  static constexpr int RPL = 64 / NP;              // rows per load instruction
  // d = 128: 8-row tiles (two rows per lane).  Each wait is for 4 KB of K
  // and V instead of 8 KB, and with eight query heads the per-row logits and
  // tile buffers leave room for two waves per SIMD; d = 64 keeps 16 rows
  // (two rows per lane there too)
  static constexpr int TILE = D == 128 ? 8 : 16;
  static constexpr int NL = TILE / RPL;            // rows of a tile per lane
  static constexpr int CW = kDecodeChunk;          // tokens per wave
  static constexpr int W = kDecodeWaves;
  static constexpr int RS = D + 4;
  static constexpr int PD0 = 2;                    // tiles in flight behind the current one (dense heads)
  static constexpr int SP = W * RPL * G * D;       // residual V accumulators (floats)
  static constexpr int MG = W * G * (D + 2);       // per-wave (acc, m, l) for the workgroup merge
  static constexpr int LDSF = SP > MG ? SP : MG;
  static constexpr int NPB = NP == 16 ? 4 : 3;     // log2 NP
  // the NL x G logits of a lane's rows fit one per lane of the row: the
  // softmax runs on a reduce-scatter of them (lane v << SH holds row v / G,
  // head v % G)
  static constexpr bool SCATTER = NL == 2 && NL * G <= NP;
  static constexpr int SH = SCATTER ? NPB - (G == 8 ? 4 : G == 4 ? 3 : G == 2 ? 2 : 1) : 0;
  static_assert(NL == 2 && CW % TILE == 0 && RPL * NP == 64, "shape");
};

template <int D, int G>
struct TileBuf {
  static constexpr int NL = SS<D, G>::NL;
  uint4 k[NL], v[NL];
  // residual entry of the lane in each of its rows (k = NP path): index byte and bf16 value
  uint32_t ki[NL], kv[NL], vi[NL], vv[NL];
  uint32_t tm;  // token-level residual set: the tile's word of the token mask
};

}  // namespace

// MULTI: the call has several parts (spans and the exact tail); otherwise
// part 0 is the only one, a compile-time constant, so the per-unit scalars
// load straight from fixed argument offsets with no lookup in front.
template <int D, int G, bool C8K, bool MULTI>
__global__ __launch_bounds__(256) void decode_stream_kernel(DecodeParams P) {
  using S = SS<D, G>;
  constexpr int NP = S::NP, RPL = S::RPL, TILE = S::TILE, NL = S::NL, CW = S::CW, W = S::W;
  constexpr uint32_t RB = D * 2;
  __shared__ float q_lds[D * G];                        // [c][g] fp32: residual K gathers
  __shared__ __attribute__((aligned(16))) float big[S::LDSF];  // residual V accumulators, then the merge
  auto sp = [&](int w, int cp, int g, int c) -> float& { return big[((w * RPL + cp) * G + g) * D + c]; };
  auto mg = [&](int w, int g, int c) -> float& { return big[(w * G + g) * (D + 2) + c]; };

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int slot = blockIdx.x % P.n_chunks_total;
  const int seq = blockIdx.x / P.n_chunks_total / P.hkv;
  const int rank = blockIdx.x / P.n_chunks_total % P.hkv;
  const int part = MULTI ? decode_part(P, slot) : 0;
  const int wgc = MULTI ? slot - P.part[part].base : slot;
  const bool tail = MULTI && part == P.tail_part;
  // Workgroups are dispatched in index order, and the older of the waves
  // sharing a SIMD are served first, so the heads of a sequence are taken
  // in cost order: residual heads (the most bytes per token) first, then
  // the others, each group in head order.  The per-unit values are fetched
  // together, as scalar loads, before the exit test reads them: the mode
  // bytes of the sequence's heads through their aligned words (the array is
  // 4-byte aligned and padded to a multiple of 4 bytes), every head's
  // segment offset, and the length; the start-up costs one round trip that
  // does not queue behind other waves' tile loads.  A segment offset is a
  // multiple of 256 and a mode is at most kExact; a unit that breaks either
  // reads nothing and writes a record that turns its query heads' outputs
  // into NaN.  (The exact tail of a generation has no unit arrays: its rows
  // are exact.  More than 8 KV heads keep the head order.)
  const int T = P.part[part].lens[seq];
  int head = rank;
  uint32_t mode_word = (uint32_t)kExact;
  uint64_t seg_off = 0;
  if (!tail) {
    const uint64_t u0 = ((uint64_t)seq * P.n_blocks + P.block) * P.hkv;
    const uint32_t* mw = reinterpret_cast<const uint32_t*>(P.part[part].modes);
    const uint64_t* so = P.part[part].seg_off + u0;
    if (P.hkv <= 8) {
      const uint64_t w0 = u0 >> 2, w1 = (u0 + P.hkv - 1) >> 2;
      const uint32_t a = mw[w0];
      const uint32_t b = w1 > w0 ? mw[w0 + 1] : 0u;
      const uint32_t c = w1 > w0 + 1 ? mw[w0 + 2] : 0u;
      uint64_t offs[8];
#pragma unroll
      for (int h = 0; h < 8; ++h) offs[h] = h < P.hkv ? so[h] : 0ull;
      const int sft = 8 * (int)(u0 & 3);
      const uint64_t lo = (uint64_t)a | ((uint64_t)b << 32);
      const uint64_t bytes = sft ? (lo >> sft) | ((uint64_t)c << (64 - sft)) : lo;  // mode of head h at bits 8h
      uint32_t rmask = 0;
#pragma unroll
      for (int h = 0; h < 8; ++h) rmask |= (h < P.hkv && ((bytes >> (8 * h)) & 0xE3u) == (uint64_t)kResidual) << h;
      const int nr = __builtin_popcount(rmask);
      uint32_t sel = rank < nr ? rmask : ~rmask & ((1u << P.hkv) - 1u);
      for (int i = rank < nr ? rank : rank - nr; i > 0; --i) sel &= sel - 1u;  // drop the lower set bits
      head = __builtin_ctz(sel);
      mode_word = (uint32_t)(bytes >> (8 * head));
#pragma unroll
      for (int h = 0; h < 8; ++h) seg_off = h == head ? offs[h] : seg_off;
    } else {
      const uint64_t unit = u0 + head;
      mode_word = mw[unit >> 2] >> (8 * (unit & 3));
      seg_off = so[head];
    }
  }
  const int sh = seq * P.hkv + head;   // the (sequence, KV head) of the record slots
  const uint32_t mbyte = mode_word & 0xFFu;
  const int mode = mode_of(mbyte);
  const int wg_tok0 = wgc * kDecodeWgTokens;
  const bool bad_unit = !unit_byte_ok(mbyte, P.tokres ? P.n_rates : 0) || (seg_off & 255) != 0;
  if (wg_tok0 >= T || bad_unit) {
    // no tokens here: an empty record, m = -inf, l = 0, acc = 0, since the
    // merge reads every slot; an invalid unit: m = 0, l = 1, acc = NaN, which
    // the merge carries into every output channel of the KV head's queries
    float* rec = P.ws + ((uint64_t)sh * P.n_chunks_total + slot) * G * S::RS;
    for (int i = threadIdx.x; i < G * S::RS; i += 256) {
      const int c = i % S::RS;
      rec[i] = bad_unit ? (c == D ? 0.f : c == D + 1 ? 1.f : __builtin_nanf("")) : (c == D ? -INFINITY : 0.f);
    }
    return;
  }

  const int k = P.topk;
  // residual heads hold either per-token channel entries or a token-level set
  const bool tokres = P.tokres && mode == kResidual;
  const bool resid = !P.tokres && (mode == kResidual) && k > 0;
  // FP8 caches: the shared planes and residual values of shared / residual
  // heads are E4M3 (one byte per channel); exact heads stay bf16
  const bool c8 = C8K && mode != kExact;
  const int ce = c8 ? 1 : 2;
  const uint8_t* seg = P.part[part].cache + seg_off;
  const int nb = P.bsize, ib = index_bytes(nb);
  const SegLayout L = seg_layout(mode, (uint64_t)T, D, k, 2, ce, nb);
  // bytes of the plane a tile reads: FP8 shared planes in whole 1 KB blocks
  const uint64_t dense = c8 ? coef_plane_bytes((uint64_t)T, D, 1) : (uint64_t)T * D * ce;
  const uint64_t xplane = plane_bytes(dense);  // exact planes: K of layer p at p * xplane, V at (B + p) * xplane
  const uint64_t tail_off = ((uint64_t)seq * P.hkv + head) * (uint64_t)P.tail_cap * RB;
  const auto kr = rsrc(tail ? static_cast<const uint8_t*>(P.tail_k) + tail_off
                            : seg + (mode == kExact ? (uint64_t)P.pos * xplane : L.mk), dense);
  const auto vr = rsrc(tail ? static_cast<const uint8_t*>(P.tail_v) + tail_off
                            : seg + (mode == kExact ? (uint64_t)(nb + P.pos) * xplane : L.mv), dense);
  const auto ikr = rsrc(seg + L.ik, (uint64_t)T * k * ib);
  const auto vkr = rsrc(seg + L.vk, (uint64_t)T * k * ce);
  const auto ivr = rsrc(seg + L.iv, (uint64_t)T * k * ib);
  const auto vvr = rsrc(seg + L.vv, (uint64_t)T * k * ce);
  const float w1 = P.wres[0], w2 = P.wres[1], w3 = P.wres[2];
  // token-level residual set: token mask, running counts, rows of the set's tokens
  const int ppm = unit_ppm(P.res_ppm, P.n_rates, P.rates_ppm, mbyte);
  const TokLayout Lt = tok_layout(mode, (uint64_t)T, D, ppm, 2, ce, nb);
  const uint64_t ntok = residual_token_count((uint64_t)T, ppm);
  const auto tmr = rsrc(seg + Lt.mask, (uint64_t)(T + 31) / 32 * 4);
  const auto tcr = rsrc(seg + Lt.count, ((uint64_t)(T + kTokChunk - 1) / kTokChunk + 1) * 4);
  const auto hkr = rsrc(seg + Lt.hk, ntok * (uint64_t)(nb - 1) * D * ce);
  const auto hvr = rsrc(seg + Lt.hv, ntok * (uint64_t)(nb - 1) * D * ce);
  const uint8_t* qbase = static_cast<const uint8_t*>(P.q) + ((uint64_t)seq * P.hq + (uint64_t)head * G) * RB;
  const auto qr = rsrc(qbase, (uint64_t)G * RB);

  const int rg = lane / NP, pc = lane % NP;  // row of a load, piece of the row
  // the lane's piece of every query, for the whole kernel
  uint4 qreg[G];
#pragma unroll
  for (int g = 0; g < G; ++g) qreg[g] = ld128(qr, (uint32_t)(g * RB + pc * 16));
  // the fp32 query for the residual gathers, read now and staged to LDS after
  // the first tiles have been requested (the waits are in issue order)
  constexpr int QPT = (D * G + 255) / 256;
  uint32_t qraw[QPT];
#pragma unroll
  for (int j = 0; j < QPT; ++j) {
    const uint32_t i = threadIdx.x + 256 * j;
    qraw[j] = __builtin_amdgcn_raw_buffer_load_b16(qr, i < D * G ? i * 2 : kOob, 0, 0);
  }

  // the wave's 128 consecutive tokens: its chunk of a token-level set's
  // running counts
  const int wtok0 = wg_tok0 + wave * CW;

  float m[G], l[G], acc[G][8];
  // scattered softmax state: the reference max of the lane's head and the
  // running sum of its (row, head) logit (lanes of one head share ms)
  float ms = -INFINITY, ls = 0.f;
  const int s_row = ((lane % NP) >> S::SH) / G;  // the lane's row of the two (0 or 1)
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -INFINITY;
    l[g] = 0.f;
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[g][c] = 0.f;
  }

  // The tile loop is specialised per residual flavour (RES: 0 none, 1 one
  // entry per lane (k = NP), 2 any other k, 3 a token-level set: the set's
  // tokens are masked out of the tile loop and taken afterwards in a pass of
  // their own, rebuilt in full) so that every load of a tile is
  // issued unconditionally: a tile past the wave's range takes the
  // out-of-range offset and reads zeros without touching memory.  With no
  // load behind a branch the compiler can wait for exactly the tile it needs
  // and leave the later tiles' loads in flight.
  auto run = [&](auto res_tag, auto c8_tag, auto q4_tag) {
    constexpr int RES = decltype(res_tag)::value;
    constexpr bool C8 = decltype(c8_tag)::value;  // FP8 planes and residual values
    constexpr bool Q4 = decltype(q4_tag)::value;  // block of four: uint16 codes 4c + j
    // channel and weight of a residual entry (the weight by bit masks: a
    // select chain here compiles to divergent branches)
    auto entry = [&](uint32_t ix, float& w) -> int {
      if constexpr (Q4) {
        const uint32_t j = ix & 3u;
        const uint32_t m1 = 0u - (uint32_t)(j == 1u), m2 = 0u - (uint32_t)(j == 2u), m3 = 0u - (uint32_t)(j == 3u);
        w = as_f32((as_u32(w1) & m1) | (as_u32(w2) & m2) | (as_u32(w3) & m3));
        return (int)(ix >> 2) & (D - 1);
      } else {
        w = w1;
        return (int)ix & (D - 1);
      }
    };

    constexpr int PD = (RES == 0 || RES == 3) ? S::PD0 : 1, NB = PD + 1;
    // the wave's tile t: rows from row0(t), nt of them in the sequence
    // (interleaved over the waves: 1.1% off the 8B decode step against a
    // contiguous 128 tokens a wave)
    auto row0 = [&](int t) -> int { return wg_tok0 + (t * W + wave) * TILE; };
    const int nt = wg_tok0 + wave * TILE < T
                       ? min(CW / TILE, (T - wg_tok0 - wave * TILE + W * TILE - 1) / (W * TILE))
                       : 0;

    // FP8 planes: a tile is one 1 KB block, and the lane's 16-byte slot of it
    // holds its piece of both of its rows (rows rg and rg + RPL)
    static_assert(!C8 || (TILE * D == kC8Block && NL == 2 && RPL * 2 == TILE), "FP8 tile = one block");
    auto load = [&](int t, TileBuf<D, G>& b) {
      const bool ok = t < nt;
      const uint32_t r0 = (uint32_t)row0(t);
      if constexpr (RES == 3) b.tm = __builtin_amdgcn_raw_buffer_load_b32(tmr, ok ? (r0 >> 5) * 4 : kOob, 0, 0);
      if constexpr (C8) {
        const uint4 w = ld128_stream(kr, ok ? r0 * D + lane * 16 : kOob);
        b.k[0] = make_uint4(w.x, w.y, 0u, 0u);
        b.k[1] = make_uint4(w.z, w.w, 0u, 0u);
      }
#pragma unroll
      for (int i = 0; i < NL; ++i) {
        const uint32_t row = r0 + i * RPL + rg;
        if constexpr (!C8) b.k[i] = ld128_stream(kr, ok ? row * RB + pc * 16 : kOob);
        if constexpr (RES == 1) {
          const uint32_t e = row * NP + pc;
          b.ki[i] = Q4 ? __builtin_amdgcn_raw_buffer_load_b16(ikr, ok ? e * 2 : kOob, 0, kNonTemporal)
                       : __builtin_amdgcn_raw_buffer_load_b8(ikr, ok ? e : kOob, 0, kNonTemporal);
          b.kv[i] = C8 ? __builtin_amdgcn_raw_buffer_load_b8(vkr, ok ? e : kOob, 0, kNonTemporal)
                       : __builtin_amdgcn_raw_buffer_load_b16(vkr, ok ? e * 2 : kOob, 0, kNonTemporal);
        }
      }
      if constexpr (C8) {
        const uint4 w = ld128_stream(vr, ok ? r0 * D + lane * 16 : kOob);
        b.v[0] = make_uint4(w.x, w.y, 0u, 0u);
        b.v[1] = make_uint4(w.z, w.w, 0u, 0u);
      }
#pragma unroll
      for (int i = 0; i < NL; ++i) {
        const uint32_t row = r0 + i * RPL + rg;
        if constexpr (!C8) b.v[i] = ld128_stream(vr, ok ? row * RB + pc * 16 : kOob);
        if constexpr (RES == 1) {
          const uint32_t e = row * NP + pc;
          b.vi[i] = Q4 ? __builtin_amdgcn_raw_buffer_load_b16(ivr, ok ? e * 2 : kOob, 0, kNonTemporal)
                       : __builtin_amdgcn_raw_buffer_load_b8(ivr, ok ? e : kOob, 0, kNonTemporal);
          b.vv[i] = C8 ? __builtin_amdgcn_raw_buffer_load_b8(vvr, ok ? e : kOob, 0, kNonTemporal)
                       : __builtin_amdgcn_raw_buffer_load_b16(vvr, ok ? e * 2 : kOob, 0, kNonTemporal);
        }
      }
    };

    auto compute = [&](int t, const TileBuf<D, G>& b) {
      const int r0 = row0(t);
      float s[NL][G];
#pragma unroll
      for (int i = 0; i < NL; ++i)
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const uint4 kp = C8 ? widen_e4m3(b.k[i]) : b.k[i];
          float a = 0.f;
#pragma unroll
          for (int w = 0; w < 4; ++w) a = dot2(word(kp, w), word(qreg[g], w), a);
          s[i][g] = a;
        }
      if constexpr (RES == 1) {
#pragma unroll
        for (int i = 0; i < NL; ++i) {
          float w;
          const int c = entry(b.ki[i], w);
          const float v = w * bf16_to_f32((uint16_t)(C8 ? e4m3x2_bf16<false>(b.kv[i]) : b.kv[i]));
#pragma unroll
          for (int g = 0; g < G; ++g) s[i][g] = fmaf(q_lds[c * G + g], v, s[i][g]);
        }
      } else if constexpr (RES == 2) {
#pragma unroll
        for (int i = 0; i < NL; ++i) {
          const uint32_t rc = (uint32_t)min(r0 + i * RPL + rg, T - 1);
          for (int e = pc; e < k; e += NP) {
            const uint32_t x = rc * k + e;
            float w;
            const int c = entry(Q4 ? __builtin_amdgcn_raw_buffer_load_b16(ikr, x * 2, 0, 0)
                                   : __builtin_amdgcn_raw_buffer_load_b8(ikr, x, 0, 0), w);
            const uint32_t raw = C8 ? e4m3x2_bf16<false>(__builtin_amdgcn_raw_buffer_load_b8(vkr, x, 0, 0))
                                    : __builtin_amdgcn_raw_buffer_load_b16(vkr, x * 2, 0, 0);
            const float v = w * bf16_to_f32((uint16_t)raw);
#pragma unroll
            for (int g = 0; g < G; ++g) s[i][g] = fmaf(q_lds[c * G + g], v, s[i][g]);
          }
        }
      }
      // probabilities of the lane's two rows per head as bf16 pairs (row 0
      // low), and as fp32 for the residual V entries
      uint32_t pp[G];
      float p[NL][G];
      if constexpr (S::SCATTER) {
        // Lane pc of the row ends up with the full logit of row s_row, head
        // (pc >> SH) % G, so the scale, the mask, the exp2 and the running sum
        // are taken once per logit rather than on every lane of the row.
        float a[NL * G];
#pragma unroll
        for (int i = 0; i < NL; ++i)
#pragma unroll
          for (int g = 0; g < G; ++g) a[i * G + g] = s[i][g];
        const float red = row_reduce_scatter<S::NPB>(a, lane);
        const int row = r0 + s_row * RPL + rg;
        const bool valid = row < T && (RES != 3 || ((b.tm >> (row & 31)) & 1u) == 0u);
        const float x = valid ? red * P.scale_log2 : -INFINITY;
        // The reference max moves only when some logit exceeds it by more than
        // kSlack (probabilities then stay below 2^kSlack); moving it takes the
        // head's max over the wave's rows and rescales the running sums.
        if (__ballot(x - ms > kSlack) != 0) {
          float mt = fmaxf(x, swap_half<NP>(x));
#pragma unroll
          for (int o = NP; o < 64; o <<= 1) mt = fmaxf(mt, __shfl_xor(mt, o, 64));
          const float mn = fmaxf(ms, mt);
          const float al = (ms == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(ms - mn);
          ls *= al;
          ms = mn;
#pragma unroll
          for (int g = 0; g < G; ++g) {
            // every lane of head g holds the same factor; lane g << SH is one
            const float alpha = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(al), g << S::SH));
#pragma unroll
            for (int c = 0; c < 8; ++c) acc[g][c] *= alpha;
            if constexpr (RES == 1 || RES == 2) {
#pragma unroll
              for (int cp = 0; cp < RPL; ++cp)
#pragma unroll
                for (int c = lane; c < D; c += 64) sp(wave, cp, g, c) *= alpha;
            }
          }
        }
        // masked rows: exp2(-inf) = 0; a token-level set can mask every row
        // of a tile before any logit has set the reference max, and
        // exp2(-inf - -inf) would be NaN
        const float pv = (RES == 3 && x == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(x - ms);
        ls += pv;
        const float pq = swap_half<NP>(pv);  // the same head's other row
        row_gather<S::SH>(s_row == 0 ? cvt_bf16x2(pv, pq) : cvt_bf16x2(pq, pv), pp, lane);
        if constexpr (RES == 1 || RES == 2) {
#pragma unroll
          for (int g = 0; g < G; ++g) {
            p[0][g] = bf16_lo(pp[g]);
            p[1][g] = bf16_hi(pp[g]);
          }
        }
      } else {
        float d = -INFINITY;
#pragma unroll
        for (int i = 0; i < NL; ++i) {
          const int row = r0 + i * RPL + rg;
          const bool valid = row < T && (RES != 3 || ((b.tm >> (row & 31)) & 1u) == 0u);
#pragma unroll
          for (int g = 0; g < G; ++g) {
            const float x = group_sum<NP>(s[i][g]) * P.scale_log2;
            s[i][g] = valid ? x : -INFINITY;
            d = fmaxf(d, s[i][g] - m[g]);
          }
        }
        if (__ballot(d > kSlack) != 0) {
#pragma unroll
          for (int g = 0; g < G; ++g) {
            float mt = s[0][g];
#pragma unroll
            for (int i = 1; i < NL; ++i) mt = fmaxf(mt, s[i][g]);
#pragma unroll
            for (int o = NP; o < 64; o <<= 1) mt = fmaxf(mt, __shfl_xor(mt, o, 64));
            const float mn = fmaxf(m[g], mt);
            const float alpha = (m[g] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m[g] - mn);
            l[g] *= alpha;
#pragma unroll
            for (int c = 0; c < 8; ++c) acc[g][c] *= alpha;
            if constexpr (RES == 1 || RES == 2) {
#pragma unroll
              for (int cp = 0; cp < RPL; ++cp)
#pragma unroll
                for (int c = lane; c < D; c += 64) sp(wave, cp, g, c) *= alpha;
            }
            m[g] = mn;
          }
        }
#pragma unroll
        for (int i = 0; i < NL; ++i)
#pragma unroll
          for (int g = 0; g < G; ++g) {
            if constexpr (RES == 3)
              p[i][g] = s[i][g] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(s[i][g] - m[g]);
            else
              p[i][g] = __builtin_amdgcn_exp2f(s[i][g] - m[g]);
            l[g] += p[i][g];
          }
#pragma unroll
        for (int g = 0; g < G; ++g) pp[g] = cvt_bf16x2(p[0][g], p[1][g]);
      }
      // P V over the dense plane: the lane's two rows share one dot2
      {
        const uint4 va = C8 ? widen_e4m3(b.v[0]) : b.v[0];
        const uint4 vb = C8 ? widen_e4m3(b.v[1]) : b.v[1];
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const uint32_t wa = word(va, w), wb = word(vb, w);
          const uint32_t lo = __builtin_amdgcn_perm(wb, wa, 0x05040100u);
          const uint32_t hi = __builtin_amdgcn_perm(wb, wa, 0x07060302u);
#pragma unroll
          for (int g = 0; g < G; ++g) {
            acc[g][2 * w] = dot2(lo, pp[g], acc[g][2 * w]);
            acc[g][2 * w + 1] = dot2(hi, pp[g], acc[g][2 * w + 1]);
          }
        }
      }
      // residual V entries: the lanes of one row hold distinct channels and
      // each row of a load has its own accumulator copy, so a plain
      // read-add-write never collides (masked rows add p = 0)
      if constexpr (RES == 1) {
#pragma unroll
        for (int i = 0; i < NL; ++i) {
          float w;
          const int c = entry(b.vi[i], w);
          float v = w * bf16_to_f32((uint16_t)(C8 ? e4m3x2_bf16<false>(b.vv[i]) : b.vv[i]));
          bool first = true;
          if constexpr (Q4) v = run_sum<NP>(c, v, pc, true, true, true, first);
          if (first) {
#pragma unroll
            for (int g = 0; g < G; ++g) sp(wave, rg, g, c) += p[i][g] * v;
          }
        }
      } else if constexpr (RES == 2) {
        // the lanes of a row walk the row's entries NP at a time, all lanes
        // in every step (entries past k read nothing and write nothing)
        const int steps = (k + NP - 1) / NP;
#pragma unroll
        for (int i = 0; i < NL; ++i) {
          const int row = r0 + i * RPL + rg;
          const uint32_t rc = (uint32_t)min(row, T - 1);
          for (int st = 0; st < steps; ++st) {
            const int e = st * NP + pc;
            const bool valid = e < k;
            const uint32_t x = rc * k + e;
            float w;
            const int c = entry(Q4 ? __builtin_amdgcn_raw_buffer_load_b16(ivr, valid ? x * 2 : kOob, 0, 0)
                                   : __builtin_amdgcn_raw_buffer_load_b8(ivr, valid ? x : kOob, 0, 0), w);
            const uint32_t raw = C8 ? e4m3x2_bf16<false>(__builtin_amdgcn_raw_buffer_load_b8(vvr, valid ? x : kOob, 0, 0))
                                    : __builtin_amdgcn_raw_buffer_load_b16(vvr, valid ? x * 2 : kOob, 0, 0);
            float v = w * bf16_to_f32((uint16_t)raw);
            bool first = valid;
            if constexpr (Q4) v = run_sum<NP>(c, v, pc, valid, e + 1 < k, e + 2 < k, first);
            if (first) {
#pragma unroll
              for (int g = 0; g < G; ++g) sp(wave, rg, g, c) += p[i][g] * v;
            }
          }
        }
      }
    };

    // ring of PD + 1 tile buffers: PD tiles stay in flight behind the one
    // being computed
    TileBuf<D, G> buf[NB];
#pragma unroll
    for (int i = 0; i < PD; ++i) load(i, buf[i]);
    if constexpr (RES == 1 || RES == 2) {
      for (int x = lane * 4; x < RPL * G * D; x += 256)
        *reinterpret_cast<float4*>(&sp(wave, 0, 0, x)) = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int j = 0; j < QPT; ++j) {
        const int i = threadIdx.x + 256 * j;
        if (i < D * G) q_lds[(i % D) * G + i / D] = bf16_to_f32((uint16_t)qraw[j]);
      }
      __syncthreads();  // the whole workgroup shares one unit, hence one flavour
    }
    if constexpr (RES == 0) {
      // dense heads: the wave's tiles unrolled at compile time, so every wait
      // is for exactly the tile computed next
      constexpr int NT = CW / TILE;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        if (t + PD < NT) load(t + PD, buf[(t + PD) % NB]);
        if (t < nt) compute(t, buf[t % NB]);
      }
    } else {
      for (int t = 0; t < nt; t += NB) {
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          load(t + j + PD, buf[(j + PD) % NB]);
          if (j == 0 || t + j < nt) compute(t + j, buf[j]);
        }
      }
    }

    if constexpr (S::SCATTER) {
      // back to values per head: the reference max, and on every lane its
      // row group's sum over both rows (the form the set pass and the merge take)
#pragma unroll
      for (int g = 0; g < G; ++g) m[g] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ms), g << S::SH));
      uint32_t lg[G];
      row_gather<S::SH>(__float_as_uint(ls + swap_half<NP>(ls)), lg, lane);
#pragma unroll
      for (int g = 0; g < G; ++g) l[g] = __uint_as_float(lg[g]);
    }

    if constexpr (RES == 3) {
      // The residual set's tokens among the wave's 128 consecutive tokens
      // (one chunk of the running counts; the dense walk above skipped them
      // whichever wave read their tile), RPL at a time: the lanes of row
      // group rg rebuild the rg-th one in full, K~ = M + sum_f w_f H_f and V~
      // alike, and fold it into the online softmax.
      constexpr int NF = Q4 ? 3 : 1;
      static_assert(CW == kTokChunk, "one count per wave");
      const uint32_t tw = (uint32_t)wtok0 >> 5;
      const bool in_a = wtok0 < T, in_b = wtok0 + 64 < T;
      const uint32_t wa = __builtin_amdgcn_raw_buffer_load_b32(tmr, in_a ? (tw + (lane >> 5)) * 4 : kOob, 0, 0);
      const uint32_t wb = __builtin_amdgcn_raw_buffer_load_b32(tmr, in_b ? (tw + 2 + (lane >> 5)) * 4 : kOob, 0, 0);
      const uint32_t base = __builtin_amdgcn_raw_buffer_load_b32(tcr, in_a ? ((uint32_t)wtok0 / kTokChunk) * 4 : kOob,
                                                                 0, 0);
      const bool bit_a = (wa >> (lane & 31)) & 1u, bit_b = (wb >> (lane & 31)) & 1u;
      const uint64_t ba = __ballot(bit_a), bb = __ballot(bit_b);
      const int na = __builtin_popcountll(ba), nres = na + __builtin_popcountll(bb);
      int* lst = reinterpret_cast<int*>(big) + wave * CW;  // wave-private (this flavour has no V accumulators)
      const uint64_t below = (1ull << lane) - 1ull;
      if (bit_a) lst[__builtin_popcountll(ba & below)] = lane;
      if (bit_b) lst[na + __builtin_popcountll(bb & below)] = 64 + lane;
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      __builtin_amdgcn_wave_barrier();
      const float wf[3] = {w1, w2, w3};
      for (int j0 = 0; j0 < nres; j0 += RPL) {
        const int j = j0 + rg;
        const bool ok = j < nres;
        const uint32_t row = (uint32_t)(wtok0 + (ok ? lst[j] : 0));
        const uint32_t hrow = (base + (uint32_t)j) * NF * D;  // element index of the token's first row
        uint4 mk, mv, hk[NF], hv[NF];
        if constexpr (C8) {
          const uint32_t o8 = (uint32_t)c8_piece_offset(row, pc, D);
          const auto a = __builtin_amdgcn_raw_buffer_load_b64(kr, ok ? o8 : kOob, 0, 0);
          const auto b2 = __builtin_amdgcn_raw_buffer_load_b64(vr, ok ? o8 : kOob, 0, 0);
          mk = widen_e4m3(make_uint4(a[0], a[1], 0u, 0u));
          mv = widen_e4m3(make_uint4(b2[0], b2[1], 0u, 0u));
#pragma unroll
          for (int f = 0; f < NF; ++f) {
            const uint32_t e = hrow + f * D + pc * 8;
            const auto x = __builtin_amdgcn_raw_buffer_load_b64(hkr, ok ? e : kOob, 0, 0);
            const auto y = __builtin_amdgcn_raw_buffer_load_b64(hvr, ok ? e : kOob, 0, 0);
            hk[f] = widen_e4m3(make_uint4(x[0], x[1], 0u, 0u));
            hv[f] = widen_e4m3(make_uint4(y[0], y[1], 0u, 0u));
          }
        } else {
          mk = ld128(kr, ok ? row * RB + pc * 16 : kOob);
          mv = ld128(vr, ok ? row * RB + pc * 16 : kOob);
#pragma unroll
          for (int f = 0; f < NF; ++f) {
            const uint32_t e = (hrow + f * D + pc * 8) * 2;
            hk[f] = ld128(hkr, ok ? e : kOob);
            hv[f] = ld128(hvr, ok ? e : kOob);
          }
        }
        float kf[8], vf[8];
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          const int w = c >> 1;
          auto ch = [&](const uint4& v) { return (c & 1) ? bf16_hi(word(v, w)) : bf16_lo(word(v, w)); };
          kf[c] = ch(mk);
          vf[c] = ch(mv);
#pragma unroll
          for (int f = 0; f < NF; ++f) {
            kf[c] = fmaf(wf[f], ch(hk[f]), kf[c]);
            vf[c] = fmaf(wf[f], ch(hv[f]), vf[c]);
          }
        }
        float sres[G];
        float dmax = -INFINITY;
#pragma unroll
        for (int g = 0; g < G; ++g) {
          float a = 0.f;
#pragma unroll
          for (int c = 0; c < 8; ++c) {
            const uint32_t qw = word(qreg[g], c >> 1);
            a = fmaf(kf[c], (c & 1) ? bf16_hi(qw) : bf16_lo(qw), a);
          }
          sres[g] = ok ? group_sum<NP>(a) * P.scale_log2 : -INFINITY;
          dmax = fmaxf(dmax, sres[g] - m[g]);
        }
        if (__ballot(dmax > kSlack) != 0) {
#pragma unroll
          for (int g = 0; g < G; ++g) {
            float mt = sres[g];
#pragma unroll
            for (int o = NP; o < 64; o <<= 1) mt = fmaxf(mt, __shfl_xor(mt, o, 64));
            const float mn = fmaxf(m[g], mt);
            const float alpha = (m[g] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m[g] - mn);
            l[g] *= alpha;
#pragma unroll
            for (int c = 0; c < 8; ++c) acc[g][c] *= alpha;
            m[g] = mn;
          }
        }
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const float pg = __builtin_amdgcn_exp2f(sres[g] - m[g]);  // rows past the set: exp2(-inf) = 0
          l[g] += pg;
#pragma unroll
          for (int c = 0; c < 8; ++c) acc[g][c] = fmaf(pg, vf[c], acc[g][c]);
        }
      }
    }
  };  // run

  using R0 = std::integral_constant<int, 0>;
  using R1 = std::integral_constant<int, 1>;
  using R2 = std::integral_constant<int, 2>;
  using R3 = std::integral_constant<int, 3>;
  using F = std::false_type;
  using Tr = std::true_type;
  // residual heads: one entry per lane of a row (k = NP) or any other k, by block size
  auto run_res = [&](auto c8_tag) {
    if (nb == 4) {
      if (k == NP)
        run(R1{}, c8_tag, Tr{});
      else
        run(R2{}, c8_tag, Tr{});
    } else {
      if (k == NP)
        run(R1{}, c8_tag, F{});
      else
        run(R2{}, c8_tag, F{});
    }
  };
  auto run_tok = [&](auto c8_tag) {
    if (nb == 4)
      run(R3{}, c8_tag, Tr{});
    else
      run(R3{}, c8_tag, F{});
  };
  if constexpr (C8K) {
    if (c8) {
      if (resid)
        run_res(Tr{});
      else if (tokres)
        run_tok(Tr{});
      else
        run(R0{}, Tr{}, F{});
    } else {
      run(R0{}, F{}, F{});  // exact heads
    }
  } else {
    if (resid)
      run_res(F{});
    else if (tokres)
      run_tok(F{});
    else
      run(R0{}, F{}, F{});
  }

  // wave totals: the row groups of a load saw different rows
#pragma unroll
  for (int o = NP; o < 64; o <<= 1)
#pragma unroll
    for (int g = 0; g < G; ++g) {
      l[g] += __shfl_xor(l[g], o, 64);
#pragma unroll
      for (int c = 0; c < 8; ++c) acc[g][c] += __shfl_xor(acc[g][c], o, 64);
    }
  if (resid && lane < NP) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int c = 0; c < 8; ++c)
#pragma unroll
        for (int cp = 0; cp < RPL; ++cp) acc[g][c] += sp(wave, cp, g, lane * 8 + c);
  }
  __syncthreads();  // the accumulator copies are read; the merge reuses their space
  if (lane < NP) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int c = 0; c < 8; ++c) mg(wave, g, lane * 8 + c) = acc[g][c];
  }
  if (lane == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      mg(wave, g, D) = m[g];
      mg(wave, g, D + 1) = l[g];
    }
  }
  __syncthreads();
  float* rec = P.ws + ((uint64_t)sh * P.n_chunks_total + slot) * G * S::RS;
  for (int i = threadIdx.x; i < G * (D + 2); i += 256) {
    const int g = i / (D + 2), c = i - g * (D + 2);
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < W; ++w) M = fmaxf(M, mg(w, g, D));
    float o;
    if (c == D) {
      o = M;
    } else {
      o = 0.f;
#pragma unroll
      for (int w = 0; w < W; ++w) {
        const float mw = mg(w, g, D);
        const float f = (mw == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mw - M);
        o = fmaf(f, mg(w, g, c), o);
      }
    }
    rec[g * S::RS + c] = o;
  }
}

// Wave-wide max / sum: DPP within each row of 16 lanes, then the four row
// results read as uniform values.
__device__ __forceinline__ float wave_max_dpp(float x) {
  x = fmaxf(x, dpp<kDppQuadXor1>(x));
  x = fmaxf(x, dpp<kDppQuadXor2>(x));
  x = fmaxf(x, dpp<kDppRowHalfMirror>(x));
  x = fmaxf(x, dpp<kDppRowMirror>(x));
  const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
  const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
  const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
  const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
  return fmaxf(fmaxf(a, b), fmaxf(c, d));
}
__device__ __forceinline__ float wave_sum_dpp(float x) {
  x += dpp<kDppQuadXor1>(x);
  x += dpp<kDppQuadXor2>(x);
  x += dpp<kDppRowHalfMirror>(x);
  x += dpp<kDppRowMirror>(x);
  const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
  const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
  const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
  const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
  return (a + b) + (c + d);
}

// Log-sum-exp merge of the workgroup records of one (sequence, query head),
// over every slot of the call (compressed spans, then the exact tail; a slot
// with no tokens holds an empty record, so no lengths are read first):
//   M = max_i m_i,  l = sum_i l_i 2^(m_i - M),  o = sum_i acc_i 2^(m_i - M) / l.
// One workgroup of four waves per query head, records taken in blocks of 64.
// Within a block every wave loads the (m, l) pairs (record i in lane i) and
// its share of the accumulators (record i to wave i mod 4) in one go -- the
// accumulators do not depend on the max -- then reduces M and l itself and
// weights each record with the value read from the lane that owns it.  A
// running (M, l, o) carries over between blocks; LDS adds the four waves'
// partial sums.
template <int D, bool BF16, int G>
__global__ __launch_bounds__(256) void decode_merge_kernel(DecodeParams P) {
  constexpr int RS = D + 4;
  constexpr int CPL = D / 64;  // channels per lane
  constexpr int NR = 16;       // records per wave per block
  __shared__ float part[4][D];
  const int qh = blockIdx.x % P.hq, seq = blockIdx.x / P.hq;
  const int head = qh / G, g = qh % G;
  const uint64_t stride = (uint64_t)G * RS;  // floats between consecutive records of one query head
  const float* head_base = P.ws + ((uint64_t)(seq * P.hkv + head) * P.n_chunks_total) * stride + g * RS;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;

  float M = -INFINITY, lsum = 0.f, o[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) o[c] = 0.f;
  // every slot of every part holds a record (empty ones have m = -inf), so
  // the slots are merged as one range without reading the lengths first
  {
    const int nch = P.n_chunks_total;
    const float* base = head_base;
  for (int b0 = 0; b0 < nch; b0 += 64) {
    const int last = nch - 1;  // loads past the end repeat the last record and get weight 0
    const int il = b0 + lane;
    const float2 ml = *reinterpret_cast<const float2*>(base + (uint64_t)min(il, last) * stride + D);
    float a[NR][CPL];
#pragma unroll
    for (int j = 0; j < NR; ++j) {
      const float* r = base + (uint64_t)min(b0 + wave + 4 * j, last) * stride;
#pragma unroll
      for (int c = 0; c < CPL; ++c) a[j][c] = r[lane * CPL + c];
    }
    const float mi = il < nch ? ml.x : -INFINITY;
    const float Mb = wave_max_dpp(mi);
    const float Mn = fmaxf(M, Mb);
    const float fo = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(M - Mn);
    const float w = (il < nch && mi != -INFINITY) ? __builtin_amdgcn_exp2f(mi - Mn) : 0.f;
    lsum = lsum * fo + wave_sum_dpp(w * ml.y);
#pragma unroll
    for (int c = 0; c < CPL; ++c) o[c] *= fo;
#pragma unroll
    for (int j = 0; j < NR; ++j) {
      const float wj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w), wave + 4 * j));
#pragma unroll
      for (int c = 0; c < CPL; ++c) o[c] = fmaf(wj, a[j][c], o[c]);
    }
    M = Mn;
  }
  }
#pragma unroll
  for (int c = 0; c < CPL; ++c) part[wave][lane * CPL + c] = o[c];
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const int ch = lane * CPL + c;
      const float s = (part[0][ch] + part[1][ch]) + (part[2][ch] + part[3][ch]);
      const float res = lsum > 0.f ? s / lsum : 0.f;
      const uint64_t oi = ((uint64_t)seq * P.hq + qh) * D + ch;
      if constexpr (BF16)
        reinterpret_cast<uint16_t*>(P.out)[oi] = (uint16_t)f32_to_bf16_bits(res);
      else
        reinterpret_cast<float*>(P.out)[oi] = res;
    }
  }
}

template <int D, int G>
static hipError_t launch_t(const DecodeParams& P, hipStream_t s) {
  const dim3 grid((unsigned)P.batch * P.hkv * P.n_chunks_total);
  const bool multi = P.n_parts > 1 || P.tail_part >= 0;
  if (P.coef8) {
    if (multi)
      hipLaunchKernelGGL((decode_stream_kernel<D, G, true, true>), grid, dim3(256), 0, s, P);
    else
      hipLaunchKernelGGL((decode_stream_kernel<D, G, true, false>), grid, dim3(256), 0, s, P);
  } else {
    if (multi)
      hipLaunchKernelGGL((decode_stream_kernel<D, G, false, true>), grid, dim3(256), 0, s, P);
    else
      hipLaunchKernelGGL((decode_stream_kernel<D, G, false, false>), grid, dim3(256), 0, s, P);
  }
  return hipGetLastError();
}

hipError_t launch_decode_stream(const DecodeParams& P, hipStream_t s) {
  if (P.n_chunks_total <= 0) return hipSuccess;
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
    case 1: hipLaunchKernelGGL((decode_merge_kernel<D, BF16, 1>), grid, dim3(256), 0, s, P); break;
    case 2: hipLaunchKernelGGL((decode_merge_kernel<D, BF16, 2>), grid, dim3(256), 0, s, P); break;
    case 4: hipLaunchKernelGGL((decode_merge_kernel<D, BF16, 4>), grid, dim3(256), 0, s, P); break;
    default: hipLaunchKernelGGL((decode_merge_kernel<D, BF16, 8>), grid, dim3(256), 0, s, P); break;
  }
  return hipGetLastError();
}

hipError_t launch_decode_merge(const DecodeParams& P, hipStream_t s) {
  if (P.d == 128) return P.bf16 ? launch_merge_d<128, true>(P, s) : launch_merge_d<128, false>(P, s);
  return P.bf16 ? launch_merge_d<64, true>(P, s) : launch_merge_d<64, false>(P, s);
}

}  // namespace fdkv
