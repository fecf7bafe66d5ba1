// Online routing probe: the logit-reconstruction loss of Eq. (2).
//
// For a (pair b, KV head h) unit, let Delta_t be K^(m)_t - K_t of one layer
// of the pair.  With B = 2 the shared reconstruction misses -D_t for layer
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
// Kernels: residual_select (compress.hip) writes every unit's K top-k channel
// indices; probe_qgram forms S_u in fp32; probe_dgram streams the key pairs,
// stages bf16(D) and bf16(Dbar) transposed in LDS and accumulates the upper
// triangle of both Gram matrices with v_mfma_f32_32x32x16_bf16 (one wave
// per matrix), then contracts them with S_u in its epilogue; probe_finalize
// sums the per-workgroup partials in a fixed order in fp64.
#include "fdkv_common.h"
#include "fdkv_kernels.h"

namespace fdkv {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

template <int D, bool BF16>
__device__ __forceinline__ float load_q(const void* base, uint64_t i) {
  if constexpr (BF16)
    return bf16_to_f32(static_cast<const uint16_t*>(base)[i]);
  else
    return static_cast<const float*>(base)[i];
}

// S_u = sum of q q^T over the probe rows of both layers and the G query heads.
template <int D, bool BF16>
__global__ __launch_bounds__(256) void probe_qgram_kernel(ProbeParams P) {
  constexpr int BS = D / 16;  // each thread owns a BS x BS block of S
  constexpr int RT = 32;      // rows per LDS tile
  __shared__ float rows[RT][D];
  const int unit = blockIdx.x;
  const int pair = unit / P.hkv, head = unit % P.hkv;
  const int G = P.hq / P.hkv, NP = P.n_probe;
  const int NR = 2 * G * NP;
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
        v = load_q<D, BF16>(P.qp[2 * pair + ls], ((uint64_t)(head * G + g) * NP + p) * D + c);
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
  float* S = P.gram_q + (uint64_t)unit * D * D;
#pragma unroll
  for (int i = 0; i < BS; ++i)
#pragma unroll
    for (int j = 0; j < BS; ++j) S[(bi + i) * D + bj + j] = acc[i][j];
}

template <int D, bool BF16>
__global__ __launch_bounds__(128) void probe_dgram_kernel(ProbeParams P) {
  constexpr int E = BF16 ? 2 : 4;
  constexpr int NP = D * E / 16;     // input pieces per row
  constexpr int CPP = 16 / E;        // channels per piece
  constexpr int NB = D / 32;         // 32-channel blocks
  constexpr int NT = NB * (NB + 1) / 2;
  constexpr int TS = kProbeStep;
  constexpr int LDT = TS + 8;        // LDS row stride in bf16 elements
  __shared__ __attribute__((aligned(16))) uint16_t dt[2][D][LDT];  // [shared/residual][channel][token]

  const int unit = blockIdx.y, chunk = blockIdx.x;
  const int pair = unit / P.hkv, head = unit % P.hkv;
  const int T = P.seq_len, k = P.topk;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const uint64_t RB = (uint64_t)D * E;
  const uint8_t* ka = static_cast<const uint8_t*>(P.k[2 * pair]) + (uint64_t)head * T * RB;
  const uint8_t* kb = static_cast<const uint8_t*>(P.k[2 * pair + 1]) + (uint64_t)head * T * RB;
  const uint8_t* idx = P.idx + (uint64_t)unit * plane_bytes((uint64_t)T * k);
  const int t_begin = chunk * kProbeChunk;
  const int t_end = min(T, t_begin + kProbeChunk);

  f32x16_t acc[NT];
#pragma unroll
  for (int i = 0; i < NT; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;

  for (int t0 = t_begin; t0 < t_end; t0 += TS) {
    // bf16(D) of TS tokens into both planes, transposed to [channel][token]
    const int piece = tid % NP;
    for (int r = tid / NP; r < TS; r += 128 / NP) {
      const int t = t0 + r;
      uint16_t h[CPP];
      if (t < t_end) {
        const uint64_t off = (uint64_t)t * RB + piece * 16;
        const uint4 a = *reinterpret_cast<const uint4*>(ka + off);
        const uint4 b = *reinterpret_cast<const uint4*>(kb + off);
        const uint32_t* pa = reinterpret_cast<const uint32_t*>(&a);
        const uint32_t* pb = reinterpret_cast<const uint32_t*>(&b);
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          if constexpr (BF16) {
            h[2 * w] = (uint16_t)f32_to_bf16_bits((bf16_lo(pa[w]) - bf16_lo(pb[w])) * 0.5f);
            h[2 * w + 1] = (uint16_t)f32_to_bf16_bits((bf16_hi(pa[w]) - bf16_hi(pb[w])) * 0.5f);
          } else {
            h[w] = (uint16_t)f32_to_bf16_bits((as_f32(pa[w]) - as_f32(pb[w])) * 0.5f);
          }
        }
      } else {
#pragma unroll
        for (int c = 0; c < CPP; ++c) h[c] = 0;
      }
#pragma unroll
      for (int c = 0; c < CPP; ++c) {
        dt[0][piece * CPP + c][r] = h[c];
        dt[1][piece * CPP + c][r] = h[c];
      }
    }
    __syncthreads();
    // residual plane: zero each token's top-k channels
    if (tid < TS) {
      const int t = t0 + tid;
      if (t < t_end)
        for (int j = 0; j < k; ++j) {
          const int c = idx[(uint64_t)t * k + j];
          if (c < D) dt[1][c][tid] = 0;
        }
    }
    __syncthreads();
    // C += Dt Dt^T on the upper-triangular 32x32 tiles, wave w on plane w
#pragma unroll
    for (int kk = 0; kk < TS / 16; ++kk) {
      bf16x8_t blk[NB];
#pragma unroll
      for (int I = 0; I < NB; ++I)
        blk[I] = *reinterpret_cast<const bf16x8_t*>(&dt[wave][32 * I + (lane & 31)][16 * kk + 8 * (lane >> 5)]);
      int ti = 0;
#pragma unroll
      for (int I = 0; I < NB; ++I)
#pragma unroll
        for (int J = I; J < NB; ++J) {
          acc[ti] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(blk[I], blk[J], acc[ti], 0, 0, 0);
          ++ti;
        }
    }
    __syncthreads();
  }

  // < C, S_u >, off-diagonal tiles counted twice (both matrices symmetric)
  const float* S = P.gram_q + (uint64_t)unit * D * D;
  float part = 0.f;
  int ti = 0;
#pragma unroll
  for (int I = 0; I < NB; ++I)
#pragma unroll
    for (int J = I; J < NB; ++J) {
      const float wgt = (I == J) ? 1.f : 2.f;
      const int col = 32 * J + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 32 * I + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        part = fmaf(wgt * acc[ti][r], S[row * D + col], part);
      }
      ++ti;
    }
  part = wave_sum(part);
  if (lane == 0) P.partial[((uint64_t)unit * P.n_chunks + chunk) * 2 + wave] = part;
}

__global__ void probe_finalize_kernel(ProbeParams P) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int units = P.n_pairs * P.hkv;
  if (i >= units * 2) return;
  const int unit = i >> 1, m = i & 1;
  double s = 0.0;
  for (int c = 0; c < P.n_chunks; ++c) s += (double)P.partial[((uint64_t)unit * P.n_chunks + c) * 2 + m];
  const int G = P.hq / P.hkv;
  P.errors[unit * 2 + m] = (float)(s / (2.0 * G * (double)P.n_probe * (double)P.d));
}

template <int D, bool BF16>
static hipError_t launch_probe_t(const ProbeParams& P, hipStream_t s) {
  const int units = P.n_pairs * P.hkv;
  hipLaunchKernelGGL((probe_qgram_kernel<D, BF16>), dim3(units), dim3(256), 0, s, P);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((probe_dgram_kernel<D, BF16>), dim3(P.n_chunks, units), dim3(128), 0, s, P);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(probe_finalize_kernel, dim3((units * 2 + 255) / 256), dim3(256), 0, s, P);
  return hipGetLastError();
}

hipError_t launch_probe(const ProbeParams& P, hipStream_t s) {
  if (P.d == 128) return P.bf16 ? launch_probe_t<128, true>(P, s) : launch_probe_t<128, false>(P, s);
  return P.bf16 ? launch_probe_t<64, true>(P, s) : launch_probe_t<64, false>(P, s);
}

}  // namespace fdkv
