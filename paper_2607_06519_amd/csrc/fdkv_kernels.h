// Kernel parameter blocks and launchers of the HIP path (internal to libfdkv).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fdkv {

constexpr int kMaxPtrLayers = 128;  // layer pointers carried in kernel arguments
constexpr int kCompressTile = 64;   // tokens per compress_dense workgroup

struct CompressParams {
  const void* k[kMaxPtrLayers];
  const void* v[kMaxPtrLayers];
  const uint8_t* modes;        // [pairs][hkv]
  const uint64_t* seg_off;     // [pairs][hkv]
  uint8_t* cache;
  int seq_len, n_pairs, hkv, d, topk;
  bool bf16;
  bool coef8;                  // shared planes in FP8 E4M3 (bf16 inputs)
};

struct SelectParams {
  const void* k[kMaxPtrLayers];
  const void* v[kMaxPtrLayers];
  const uint8_t* modes;        // null: select every unit (probe); else residual units only
  const uint64_t* seg_off;
  uint8_t* cache;
  uint8_t* idx_out;            // probe: [units] planes of plane_bytes(T*k) bytes
  int seq_len, n_pairs, hkv, d, topk;
  bool bf16;
  bool coef8;                  // residual values in FP8 E4M3 (bf16 inputs)
};

// decode: tokens per wave and waves per workgroup of the split-K kernel
constexpr int kDecodeChunk = 128;
constexpr int kDecodeWaves = 4;
constexpr int kDecodeWgTokens = kDecodeChunk * kDecodeWaves;

struct DecodeParams {
  const uint8_t* cache;
  const uint64_t* seg_off;     // [batch][pairs][hkv]
  const uint8_t* modes;        // [batch][pairs][hkv]
  const int32_t* seq_lens;     // [batch]
  const void* q;               // [batch][hq][d]
  void* out;                   // [batch][hq][d]
  float* ws;                   // partials [batch][hkv][n_wgchunks][G][d + 4]
  int layer, n_pairs, hkv, hq, d, topk, n_wgchunks, batch;
  float scale_log2;            // sm_scale * log2(e)
  bool bf16;
  bool coef8;                  // shared planes and residual values of shared / residual heads in FP8 E4M3
};

// probe
constexpr int kProbeStep = 128;     // tokens per MFMA step
constexpr int kProbeChunk = 1024;   // tokens per probe workgroup

struct ProbeParams {
  const void* k[kMaxPtrLayers];
  const void* qp[kMaxPtrLayers];
  const uint8_t* idx;          // K residual indices per unit (from residual_select)
  float* gram_q;               // [units][d][d]  sum of q q^T over the unit's probe rows
  float* partial;              // [units][n_chunks][2]
  float* errors;               // [units][2]
  int seq_len, n_pairs, hkv, hq, d, topk, n_probe, n_chunks;
  bool bf16;
};

hipError_t launch_compress_dense(const CompressParams& P, hipStream_t s);
hipError_t launch_residual_select(const SelectParams& P, int tensors, hipStream_t s);
hipError_t launch_decode(const DecodeParams& P, hipStream_t s);
hipError_t launch_decode_stream(const DecodeParams& P, hipStream_t s);  // bf16 split-K part
hipError_t launch_decode_merge(const DecodeParams& P, hipStream_t s);   // log-sum-exp merge of the records
hipError_t launch_probe(const ProbeParams& P, hipStream_t s);

}  // namespace fdkv
