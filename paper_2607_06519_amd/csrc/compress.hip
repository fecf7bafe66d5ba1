// Prefill-time compression of the KV cache (Section 3, Eq. 1 and Eq. 3).
//
// Kernels:
//  * compress_dense - coalesced streaming pass over every (block, KV head):
//    shared/residual heads write the block mean M (the per-layer image of
//    the low-frequency DCT coefficient, the same for every layer of the
//    block) for K and V; exact heads copy the input rows.  Residual heads
//    also take their entries from the same rows, K and V independently:
//    pairs each token's top-k channels of |fl32(x[2b] - x[2b+1])|, written
//    as ascending uint8 indices plus D = (x[2b] - x[2b+1]) / 2 at those
//    channels; blocks of four the top-k of the token's 3d high-frequency
//    coefficients |Z_j[c]| of the DCT-II(4) (the fp32 butterfly of dct4.h),
//    written as ascending uint16 codes 4c + j plus Z_j[c].  Both rank with
//    the wavefront top-k of rowtopk.h (ties to the lower channel or code).
#include "fdkv_common.h"
#include "fdkv_kernels.h"
#include "fp8.h"
#include "rowtopk.h"

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
  float m[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) m[i] = block_mean<true, NB>(x, i);
  return make_uint2(e4m3_quad(m[0], m[1], m[2], m[3]), e4m3_quad(m[4], m[5], m[6], m[7]));
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

// Pieces of one token row a thread of the pairs' dense pass holds: two where
// the row then still spans at least 8 lanes (fewer count reductions per
// bisection step of the top-k, more rows per wave), else one.  Lane lr of a
// row holds pieces h LPR + lr, h < PPT, so that the row's lanes load and
// store each run of LPR pieces as one contiguous span.  Blocks of four keep
// one piece (3 CPP keys a lane already).
template <int D, bool BF16, int NB>
struct DenseLayout {
  static constexpr int E = BF16 ? 2 : 4;
  static constexpr int NP = D * E / 16;               // 16-byte pieces per row
  static constexpr int PPT = (NB == 2 && NP >= 16) ? 2 : 1;
  static constexpr int LPR = NP / PPT;                // lanes per row
  static constexpr int RPP = 256 / LPR;               // rows per pass of 256 threads
  static constexpr int RPW = 64 / LPR;                // rows of a pass per wave
};

// Residual entries of pairs, from the rows the dense pass holds: the lanes
// of a token row find its top-k channels of |fl32(a - b)| (row_topk_mask),
// each lane puts its selected channels and their half differences D at
// their slots (the row's selected channels in ascending order: those of the
// row's earlier runs of pieces, then the lanes' counts before it in its run,
// then its own order) into the wave's LDS staging, and the wave writes its
// rows' index and value runs with 4-byte stores (bytes where a run does not
// start on a 4-byte boundary, and for its last partial word).
// x[h][n]: piece h LPR + lr of layer n (lr: the lane's place in the row), so
// key h CPP + c is channel CPP (h LPR + lr) + c.  PRESET: the lane's
// selection is `preset` (the probe's, of the same keys, so the same
// channels), and no keys are formed.
template <int D, bool BF16, bool C8, bool PRESET = false>
__device__ __forceinline__ void residual_entries(const uint4 (&x)[DenseLayout<D, BF16, 2>::PPT][2], int k,
                                                 int row_in_wave, int t0w, int T, uint8_t* idx_plane,
                                                 uint8_t* val_plane, uint8_t* stage, uint32_t preset = 0) {
  using Ly = DenseLayout<D, BF16, 2>;
  constexpr int E = Ly::E, CPP = 16 / E, PPT = Ly::PPT, LPR = Ly::LPR, RPW = Ly::RPW, KPT = PPT * CPP;
  constexpr int VB = C8 ? 1 : E;                       // bytes per stored value
  uint32_t key[KPT];
  float dv[KPT];
#pragma unroll
  for (int h = 0; h < PPT; ++h)
#pragma unroll
    for (int c = 0; c < CPP; ++c) {
      const float df = chan<BF16>(x[h][0], c) - chan<BF16>(x[h][1], c);
      if constexpr (!PRESET) key[h * CPP + c] = as_u32(df) & 0x7FFFFFFFu;
      dv[h * CPP + c] = df * 0.5f;
    }
  uint32_t sel = preset;
  if constexpr (!PRESET) sel = row_topk_mask<LPR, KPT, PPT>(key, k);
  // bf16 values: every channel's rounded half difference, one conversion per pair
  uint32_t hv[KPT / 2];
  if constexpr (BF16 && !C8) {
#pragma unroll
    for (int c = 0; c < KPT / 2; ++c) hv[c] = cvt_bf16x2(dv[2 * c], dv[2 * c + 1]);
  }
  const int lr = (int)(threadIdx.x & (LPR - 1));
  // staging of the wave: RPW rows x k index bytes, then RPW rows x k values
  uint8_t* si = stage;
  uint8_t* sv = stage + ((RPW * k + 3) & ~3);
  // the slot of the lane's first selected channel of each piece; the others
  // follow it
  int e0[PPT];
  uint32_t base = 0;
#pragma unroll
  for (int h = 0; h < PPT; ++h) {
    const uint32_t mine = (uint32_t)__builtin_popcount((sel >> (h * CPP)) & ((1u << CPP) - 1u));
    e0[h] = row_in_wave * k + (int)(base + row_prefix_u32<LPR>(mine) - mine);
    if (h + 1 < PPT) base += row_sum_u32<LPR>(mine);
  }
#pragma unroll
  for (int c = 0; c < KPT; ++c) {
    if ((sel >> c) & 1u) {
      const int h = c / CPP, cc = c % CPP;
      const int e = e0[h] + __builtin_popcount((sel >> (h * CPP)) & ((1u << cc) - 1u));
      si[e] = (uint8_t)((h * LPR + lr) * CPP + cc);
      if constexpr (C8)
        sv[e] = e4m3_one(dv[c]);
      else if constexpr (BF16)
        reinterpret_cast<uint16_t*>(sv)[e] = (uint16_t)(hv[c >> 1] >> (16 * (c & 1)));
      else
        reinterpret_cast<float*>(sv)[e] = dv[c];
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const int lane = (int)(threadIdx.x & 63);
  const int rows = max(0, min(RPW, T - t0w));
  auto copy = [&](const uint8_t* src, uint8_t* dst, int nbytes) {
    // 4-byte stores where the run starts on a 4-byte boundary, bytes otherwise
    const int nw = (reinterpret_cast<uintptr_t>(dst) & 3) == 0 ? nbytes >> 2 : 0;
    for (int i = lane; i < nw; i += 64)
      *reinterpret_cast<uint32_t*>(dst + 4 * i) = *reinterpret_cast<const uint32_t*>(src + 4 * i);
    for (int i = 4 * nw + lane; i < nbytes; i += 64) dst[i] = src[i];
  };
  copy(si, idx_plane + (uint64_t)t0w * k, rows * k);
  copy(sv, val_plane + (uint64_t)t0w * k * VB, rows * k * VB);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();  // the staging is free for the next rows
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Residual entries of blocks of four, from the rows the dense pass holds: each
// lane evaluates the fp32 butterfly (dct4.h) of its CPP channels, keys the 3
// CPP coefficients |Z_j[c]| in code order (bit 3 c + j - 1), finds the row's
// top-k (row_topk_mask: ties to the lower code), and stages its selected
// codes 4c + j (uint16) and coefficients at consecutive slots of the wave's
// LDS area, which the wave then writes with 4-byte stores like the pairs.
template <int D, bool BF16, bool C8>
__device__ __forceinline__ void residual_entries4(const uint4 (&x)[4], int k, int row_in_wave, int t0w, int T,
                                                  uint8_t* idx_plane, uint8_t* val_plane, uint8_t* stage,
                                                  const uint32_t* preset = nullptr) {
  constexpr int E = BF16 ? 2 : 4;
  constexpr int NP = D * E / 16, CPP = 16 / E, NK = 3 * CPP, RPW = 64 / NP;
  constexpr int VB = C8 ? 1 : E;
  uint32_t sel;
  if (preset) {  // the probe's selection of this row (the same keys, so the same coefficients)
    sel = *preset;
  } else {
    uint32_t key[NK];
#pragma unroll
    for (int c = 0; c < CPP; ++c) {
      float z[3];
      dct4_high(chan<BF16>(x[0], c), chan<BF16>(x[1], c), chan<BF16>(x[2], c), chan<BF16>(x[3], c), z[0], z[1],
                z[2]);
#pragma unroll
      for (int j = 0; j < 3; ++j) key[3 * c + j] = as_u32(z[j]) & 0x7FFFFFFFu;
    }
    sel = row_topk_mask<NP, NK>(key, k);
  }
  // the staging below evaluates the butterfly again rather than keep its NK
  // results alive (an empty asm statement that only marks the input pieces
  // as possibly changed)
  uint4 y[4] = {x[0], x[1], x[2], x[3]};
#pragma unroll
  for (int n = 0; n < 4; ++n) asm volatile("" : "+v"(y[n].x), "+v"(y[n].y), "+v"(y[n].z), "+v"(y[n].w));
  const uint32_t mine = (uint32_t)__builtin_popcount(sel);
  const uint32_t incl = row_prefix_u32<NP>(mine);
  const int lr = (int)(threadIdx.x & (NP - 1));
  uint16_t* si = reinterpret_cast<uint16_t*>(stage);
  uint8_t* sv = stage + ((RPW * k * 2 + 3) & ~3);
  const int e0 = row_in_wave * k + (int)(incl - mine);
#pragma unroll
  for (int c = 0; c < CPP; ++c) {
    if (((sel >> (3 * c)) & 7u) == 0u) continue;
    float z[3];  // evaluated again (the same rounded operations): fewer live registers
    dct4_high(chan<BF16>(y[0], c), chan<BF16>(y[1], c), chan<BF16>(y[2], c), chan<BF16>(y[3], c), z[0], z[1],
              z[2]);
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      const int b = 3 * c + j;
      if ((sel >> b) & 1u) {
        const int e = e0 + __builtin_popcount(sel & ((1u << b) - 1u));
        si[e] = (uint16_t)(4 * (lr * CPP + c) + j + 1);
        if constexpr (C8)
          sv[e] = e4m3_one(z[j]);
        else if constexpr (BF16)
          reinterpret_cast<uint16_t*>(sv)[e] = (uint16_t)f32_to_bf16_bits(z[j]);
        else
          reinterpret_cast<float*>(sv)[e] = z[j];
      }
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const int lane = (int)(threadIdx.x & 63);
  const int rows = max(0, min(RPW, T - t0w));
  auto copy = [&](const uint8_t* src, uint8_t* dst, int nbytes) {
    const int nw = (reinterpret_cast<uintptr_t>(dst) & 3) == 0 ? nbytes >> 2 : 0;
    for (int i = lane; i < nw; i += 64)
      *reinterpret_cast<uint32_t*>(dst + 4 * i) = *reinterpret_cast<const uint32_t*>(src + 4 * i);
    for (int i = 4 * nw + lane; i < nbytes; i += 64) dst[i] = src[i];
  };
  copy(stage, idx_plane + (uint64_t)t0w * k * 2, rows * k * 2);
  copy(sv, val_plane + (uint64_t)t0w * k * VB, rows * k * VB);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();  // the staging is free for the next rows
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Waves per SIMD: four for pairs (128 VGPRs with K and V taken in turn),
// three for blocks of four.  Left to itself the compiler gives blocks of
// four with bf16 inputs 180 VGPRs (two waves); held to 168 they spill three
// and the mixed 8B prefill compress takes 2.15 instead of 2.68 ms (held to
// 128 they spill 31 and take 2.58 ms).
template <int D, bool BF16, int NB>
__global__ __launch_bounds__(256, NB == 2 ? 4 : 3) void compress_dense_kernel(CompressParams P) {
  using Ly = DenseLayout<D, BF16, NB>;
  constexpr int E = Ly::E;
  constexpr int PPT = Ly::PPT, LPR = Ly::LPR;  // a thread: pieces h LPR + lr, h < PPT, of a row
  constexpr int RPP = Ly::RPP;          // rows per pass
  constexpr int RPW = Ly::RPW;          // rows of a pass per wave
  static_assert(kCompressTile % RPP == 0, "passes per tile");
  // per wave: RPW rows x (k indices of up to 2 bytes + k values of up to 4 bytes)
  __shared__ __attribute__((aligned(16))) uint8_t stage[4][RPW * D * 6 + 16];
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
  const int lr = threadIdx.x % LPR;
  const int row0 = blockIdx.x * kCompressTile + threadIdx.x / LPR;
  // residual heads with per-token channel (pairs) or coefficient (fours)
  // entries take them in this pass too
  const bool resid = mode == kResidual && !P.tokres && P.topk > 0;
  // FP8 shared planes fill whole 1 KB blocks of R8 rows: the rows after the
  // last token of its block are written as zeros, so that a decode tile (one
  // block) reads no stale bytes (R8 divides the rows of a pass, so they lie
  // in the pass of the last token)
  constexpr int R8 = kC8Block / D;
  const bool pad8 = c8 && mode != kExact;
  const int t_end = pad8 ? (T + R8 - 1) / R8 * R8 : T;
  static_assert(RPP % R8 == 0 || !BF16, "FP8 blocks within a pass");
#pragma unroll 2
  for (int r = 0; r < kCompressTile; r += RPP) {
    const int t = row0 + r;
    // rows past the end: the residual pass needs every lane of a wave, so a
    // workgroup with residual rows runs the pass to the end on zeros and
    // stores nothing for them (but the FP8 block padding)
    if (!resid && t >= t_end) break;
    if (resid && blockIdx.x * kCompressTile + r >= T) break;
    const bool live = t < T;
    uint4 ka[PPT][NB], va[PPT][NB];
    // a tensor's rows of the pass (pairs)
    auto load_rows = [&](const uint8_t* const* x, uint4 (&a)[PPT][NB]) {
#pragma unroll
      for (int h = 0; h < PPT; ++h) {
        const uint64_t off = (uint64_t)t * row_bytes + (h * LPR + lr) * 16;
#pragma unroll
        for (int n = 0; n < NB; ++n) a[h][n] = live ? load_stream(x[n] + off) : make_uint4(0u, 0u, 0u, 0u);
      }
    };
    // the planes' stores of piece h LPR + lr of one tensor of a pair (called
    // once per piece: around these stores a loop, even of one trip, gave the
    // register allocation more VGPRs)
    auto store_piece = [&](const int h, const uint4 (&a)[PPT][NB], const uint64_t mplane, const uint64_t* eplane) {
      const int piece = h * LPR + lr;
      const uint64_t off = (uint64_t)t * row_bytes + piece * 16;
      if (!live) {
        if (pad8 && t < t_end) {
          const uint64_t o8 = c8_piece_offset((uint64_t)t, piece, D);
          *reinterpret_cast<uint2*>(seg + mplane + o8) = make_uint2(0u, 0u);
        }
      } else if (mode == kExact) {
#pragma unroll
        for (int n = 0; n < NB; ++n) store_stream(seg + eplane[n] + off, a[h][n]);
      } else if (c8) {
        const uint64_t o8 = c8_piece_offset((uint64_t)t, piece, D);  // the 1 KB block layout of FP8 planes
        *reinterpret_cast<uint2*>(seg + mplane + o8) = mean_piece_e4m3<NB>(a[h]);
      } else {
        store_stream(seg + mplane + off, mean_piece<BF16, NB>(a[h]));
      }
    };
    static_assert(PPT <= 2, "pieces per thread");
    static_assert(PPT == 1 || NB == 2, "blocks of four: one piece a thread");
    const int wave = threadIdx.x >> 6;
    const int t0w = blockIdx.x * kCompressTile + r + wave * RPW;
    const int rw = (threadIdx.x & 63) / LPR;
    if constexpr (NB == 2) {
      // pairs: K, then V (a tensor's rows load, store their planes and, for
      // residual heads, their entries before the other tensor's rows load;
      // both tensors' rows in flight together took 150 VGPRs, or 128 with
      // spills whose scratch writes reached HBM); residual heads are uniform
      // over the workgroup (one unit) and every lane of a row takes part;
      // K's entries take the probe's selection of the row's pieces when
      // given (rows past the end take 0)
      // V's rows load with K's unless K selects its own channels first
      const bool early_v = !resid || P.ksel != nullptr;
      load_rows(kx, ka);
      if (early_v) load_rows(vx, va);
      store_piece(0, ka, L.mk, L.ek);
      if constexpr (PPT == 2) store_piece(1, ka, L.mk, L.ek);
      if (resid) {
        if (P.ksel) {
          uint32_t kpre = 0;
          if (live) {
            constexpr int CPP = 16 / E;
#pragma unroll
            for (int h = 0; h < PPT; ++h)
              kpre |= (uint32_t)P.ksel[selection_offset(unit, T, t, h * LPR + lr, D, E, P.ksel_bytes)] << (h * CPP);
          }
          if (c8)
            residual_entries<D, BF16, true, true>(ka, P.topk, rw, t0w, T, seg + L.ik, seg + L.vk, stage[wave], kpre);
          else
            residual_entries<D, BF16, false, true>(ka, P.topk, rw, t0w, T, seg + L.ik, seg + L.vk, stage[wave], kpre);
        } else {
          if (c8)
            residual_entries<D, BF16, true>(ka, P.topk, rw, t0w, T, seg + L.ik, seg + L.vk, stage[wave]);
          else
            residual_entries<D, BF16, false>(ka, P.topk, rw, t0w, T, seg + L.ik, seg + L.vk, stage[wave]);
        }
      }
      if (!early_v) load_rows(vx, va);
      store_piece(0, va, L.mv, L.ev);
      if constexpr (PPT == 2) store_piece(1, va, L.mv, L.ev);
      if (resid) {
        if (c8)
          residual_entries<D, BF16, true>(va, P.topk, rw, t0w, T, seg + L.iv, seg + L.vv, stage[wave]);
        else
          residual_entries<D, BF16, false>(va, P.topk, rw, t0w, T, seg + L.iv, seg + L.vv, stage[wave]);
      }
    } else {
      // blocks of four: both tensors' rows in flight together, both planes'
      // stores, then the entries (of the orders tried, the one that spills
      // the fewest registers at three waves per SIMD)
#pragma unroll
      for (int h = 0; h < PPT; ++h) {
        const uint64_t off = (uint64_t)t * row_bytes + (h * LPR + lr) * 16;
#pragma unroll
        for (int n = 0; n < NB; ++n) {
          ka[h][n] = live ? load_stream(kx[n] + off) : make_uint4(0u, 0u, 0u, 0u);
          va[h][n] = live ? load_stream(vx[n] + off) : make_uint4(0u, 0u, 0u, 0u);
        }
      }
      {
        const uint64_t off = (uint64_t)t * row_bytes + lr * 16;
        if (!live) {
          if (pad8 && t < t_end) {
            const uint64_t o8 = c8_piece_offset((uint64_t)t, lr, D);
            *reinterpret_cast<uint2*>(seg + L.mk + o8) = make_uint2(0u, 0u);
            *reinterpret_cast<uint2*>(seg + L.mv + o8) = make_uint2(0u, 0u);
          }
        } else if (mode == kExact) {
#pragma unroll
          for (int n = 0; n < NB; ++n) {
            store_stream(seg + L.ek[n] + off, ka[0][n]);
            store_stream(seg + L.ev[n] + off, va[0][n]);
          }
        } else if (c8) {
          const uint64_t o8 = c8_piece_offset((uint64_t)t, lr, D);
          *reinterpret_cast<uint2*>(seg + L.mk + o8) = mean_piece_e4m3<NB>(ka[0]);
          *reinterpret_cast<uint2*>(seg + L.mv + o8) = mean_piece_e4m3<NB>(va[0]);
        } else {
          store_stream(seg + L.mk + off, mean_piece<BF16, NB>(ka[0]));
          store_stream(seg + L.mv + off, mean_piece<BF16, NB>(va[0]));
        }
      }
      if (resid) {
        uint32_t kpre = 0;
        if (P.ksel && live)
          kpre = *reinterpret_cast<const uint32_t*>(P.ksel + selection_offset(unit, T, t, lr, D, E, 4));
        const uint32_t* kp = P.ksel ? &kpre : nullptr;
        if (c8) {
          residual_entries4<D, BF16, true>(ka[0], P.topk, rw, t0w, T, seg + L.ik, seg + L.vk, stage[wave], kp);
          residual_entries4<D, BF16, true>(va[0], P.topk, rw, t0w, T, seg + L.iv, seg + L.vv, stage[wave]);
        } else {
          residual_entries4<D, BF16, false>(ka[0], P.topk, rw, t0w, T, seg + L.ik, seg + L.vk, stage[wave], kp);
          residual_entries4<D, BF16, false>(va[0], P.topk, rw, t0w, T, seg + L.iv, seg + L.vv, stage[wave]);
        }
      }
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


}  // namespace fdkv
