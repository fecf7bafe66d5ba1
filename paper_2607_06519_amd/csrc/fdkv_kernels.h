// Kernel parameter blocks and launchers of the HIP path (internal to libfdkv).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fdkv_common.h"

namespace fdkv {

constexpr int kMaxPtrLayers = 128;  // layer pointers carried in kernel arguments
constexpr int kMaxBlocks = kMaxPtrLayers / 2;
constexpr int kCompressTile = 64;   // tokens per compress_dense workgroup

// The blocks one launch covers (all of one block size).  Unit arrays (modes,
// segment offsets, probe errors) are indexed by block * hkv + head.
struct BlockList {
  int n;
  int16_t block[kMaxBlocks];   // block index
  int16_t first[kMaxBlocks];   // first layer of the block
};

struct CompressParams {
  const void* k[kMaxPtrLayers];
  const void* v[kMaxPtrLayers];
  const uint8_t* modes;        // [blocks][hkv]
  const uint64_t* seg_off;     // [blocks][hkv]
  uint8_t* cache;
  BlockList bl;                // blocks of size bsize
  int seq_len, bsize, hkv, d, topk;
  bool bf16;
  bool coef8;                  // shared planes in FP8 E4M3 (bf16 inputs)
  bool tokres;                 // token-level residual set (else per-token channel top-k)
  int res_ppm;                 // its fraction of tokens, parts per million
  const float* scores;         // token scores [blocks][hkv][T] (token-level residual set)
  const uint8_t* ksel;         // the probe's K selections (selection_offset), or null
  int ksel_bytes;              // bytes per piece of ksel (1, or 4 with blocks of four)
};

// The K selections that the probe takes and compress may reuse: unit u's
// row t holds one slot of sb bytes per 16-byte input piece p at
// selection_offset(u, t, p): a pair's mask of the piece's CPP channels
// (bit i: channel CPP p + i, CPP = 16 / element bytes) in the slot's first
// byte, a block of four's mask of the piece's 3 CPP coefficients (bit
// 3 c + j - 1: Z_j of channel CPP p + c) as a 32-bit word.  sb is 4 when the
// schedule has blocks of four, else 1.
__host__ __device__ __forceinline__ uint64_t selection_pieces(int d, int elem_bytes) {
  return (uint64_t)d * elem_bytes / 16;
}
__host__ __device__ __forceinline__ uint64_t selection_offset(uint64_t unit, uint64_t T, uint64_t t, int p,
                                                             int d, int elem_bytes, int sb) {
  return ((unit * T + t) * selection_pieces(d, elem_bytes) + (uint64_t)p) * (uint64_t)sb;
}

// Token-level residual set: score kernel (probe), selection and rows.
struct TokenParams {
  const void* k[kMaxPtrLayers];
  const void* v[kMaxPtrLayers];
  const void* qp[kMaxPtrLayers];
  const uint8_t* modes;        // null: every unit (probe); else residual units only (compress)
  const uint64_t* seg_off;
  uint8_t* cache;
  float* scores;               // [blocks][hkv][T]
  float* sumsq;                // [blocks][hkv][T] (probe)
  float* errors;               // [blocks][hkv][2] (probe)
  BlockList bl;
  int seq_len, bsize, hkv, hq, d, n_probe, res_ppm;
  int n_rates;                 // routed fractions (0: every residual unit keeps res_ppm)
  int rates_ppm[kMaxRates];
  bool bf16, coef8;
};

// The fraction of tokens (parts per million) a residual unit's set keeps.
__host__ __device__ __forceinline__ int unit_ppm(int res_ppm, int n_rates, const int* rates, uint32_t byte) {
  return n_rates ? rates[rate_of(byte)] : res_ppm;
}

// decode: tokens per wave and waves per workgroup of the split-K kernel
constexpr int kDecodeChunk = 128;
constexpr int kDecodeWaves = 4;
constexpr int kDecodeWgTokens = kDecodeChunk * kDecodeWaves;
constexpr int kMaxParts = 16;       // compressed spans plus the exact tail of one decode call

// One part of a decode call (a compressed span or the exact tail); its
// fields sit together so that part 0 loads in one go.
struct DecodePart {
  const int32_t* lens;         // [batch] tokens of each sequence in the part
  const uint8_t* cache;
  const uint8_t* modes;        // [batch][blocks][hkv], 4-byte aligned
  const uint64_t* seg_off;     // [batch][blocks][hkv]
  int base, chunks;            // record slots [base, base + chunks) of each (sequence, KV head)
};

struct DecodeParams {
  const void* q;               // [batch][hq][d]
  bool tokres;                 // residual heads hold a token-level residual set
  int res_ppm;
  int n_rates;                 // routed fractions of the sets (0: every set keeps res_ppm)
  int rates_ppm[kMaxRates];
  void* out;                   // [batch][hq][d]
  float* ws;                   // records [batch][hkv][n_chunks_total][G][d + 4]
  int block, pos, bsize;       // the layer's block, its position in it, the block size
  int n_blocks, hkv, hq, d, topk, batch;
  // Parts of one call: compressed spans, then (if tail_part >= 0) the exact
  // tail.  The records of one (sequence, KV head) sit in n_chunks_total
  // slots.  One split-K launch covers every part: workgroup x is slot
  // x % n_chunks_total of (sequence, KV head) x / n_chunks_total.
  int n_parts, n_chunks_total, tail_part;
  DecodePart part[kMaxParts];
  float wres[3];               // weight of a residual entry of frequency j = 1..3 at this layer
                               // (B = 2: +-1 for the stored half difference)
  float scale_log2;            // sm_scale * log2(e)
  bool bf16;
  bool coef8;                  // shared planes and residual values of shared / residual heads in FP8 E4M3
  const void* tail_k;          // [batch][hkv][tail_cap][d] of the decoded layer
  const void* tail_v;
  int tail_cap;
};

// Part of a decode workgroup's record slot r (parts in slot order; uniform).
__device__ __forceinline__ int decode_part(const DecodeParams& P, int r) {
  int part = 0;
  while (part + 1 < P.n_parts && r >= P.part[part + 1].base) ++part;
  return part;
}

// generation: append one token's K / V rows of one layer to the exact tail
struct AppendParams {
  const int32_t* pos;          // [batch] row to write; rows outside [0, cap) are skipped
  const void* k_new;           // [batch][hkv][d]
  const void* v_new;
  void* tail_k;                // [batch][hkv][cap][d]
  void* tail_v;
  int batch, hkv, cap, row_bytes;
};

// probe
constexpr int kProbeStep = 128;     // tokens per MFMA step
constexpr int kProbeChunk = 1024;   // tokens per probe workgroup

struct ProbeParams {
  const void* k[kMaxPtrLayers];
  const void* qp[kMaxPtrLayers];
  float* gram_q;               // [layers][hkv][d][d]  sums of q q^T over probe rows (see probe.hip)
  float* partial;              // [units][n_chunks][2]
  float* errors;               // [units][2]
  uint8_t* ksel;               // out: the K selections (selection_offset), or null
  int ksel_bytes;              // bytes per piece of ksel (1, or 4 with blocks of four)
  BlockList bl;                // blocks of size bsize
  int8_t bsizes[kMaxBlocks];   // every block's size (finalize)
  int seq_len, bsize, n_blocks, hkv, hq, d, topk, n_probe, n_chunks;
  bool bf16;
};

hipError_t launch_compress_dense(const CompressParams& P, hipStream_t s);
hipError_t launch_decode(const DecodeParams& P, hipStream_t s);        // split-K over every part (bf16 or fp32)
hipError_t launch_decode_stream(const DecodeParams& P, hipStream_t s);  // bf16 split-K
hipError_t launch_decode_merge(const DecodeParams& P, hipStream_t s);   // log-sum-exp merge of the records
hipError_t launch_append(const AppendParams& P, hipStream_t s);
// counts[0] += E4M3 encoder mismatches, counts[1] += bf16 rounding mismatches
hipError_t launch_check_conversions(unsigned long long* counts, hipStream_t s);
hipError_t launch_token_scores(const TokenParams& P, hipStream_t s);   // the blocks of P.bl (one size)
hipError_t launch_token_select(const TokenParams& P, hipStream_t s);   // probe: errors; compress: mask, counts
hipError_t launch_token_rows(const TokenParams& P, hipStream_t s);     // compress: rows of the selected tokens
hipError_t launch_probe(const ProbeParams& P, hipStream_t s);           // the blocks of P.bl (one size)
hipError_t launch_probe_finalize(const ProbeParams& P, hipStream_t s);  // every unit

}  // namespace fdkv
