// Generation (Section 3, end of the method): routing is decided after
// prefill and reused while decoding, so the tokens a decode step produces
// stay exact until a refresh compresses them.  This kernel writes one
// layer's new K and V rows into that exact tail, row pos[s] of every
// (sequence s, KV head): one workgroup per (sequence, KV head), 16-byte
// pieces, coalesced.
#include "fdkv_common.h"
#include "fdkv_kernels.h"

namespace fdkv {

__global__ __launch_bounds__(64) void append_kernel(AppendParams P) {
  const int sh = blockIdx.x, seq = sh / P.hkv;
  const int pos = P.pos[seq];
  if (pos < 0 || pos >= P.cap) return;
  const uint64_t src = (uint64_t)sh * P.row_bytes;
  const uint64_t dst = ((uint64_t)sh * P.cap + pos) * P.row_bytes;
  const uint4* ks = reinterpret_cast<const uint4*>(static_cast<const uint8_t*>(P.k_new) + src);
  const uint4* vs = reinterpret_cast<const uint4*>(static_cast<const uint8_t*>(P.v_new) + src);
  uint4* kd = reinterpret_cast<uint4*>(static_cast<uint8_t*>(P.tail_k) + dst);
  uint4* vd = reinterpret_cast<uint4*>(static_cast<uint8_t*>(P.tail_v) + dst);
  for (int i = threadIdx.x; i < P.row_bytes / 16; i += 64) {
    kd[i] = ks[i];
    vd[i] = vs[i];
  }
}

hipError_t launch_append(const AppendParams& P, hipStream_t s) {
  if (P.batch * P.hkv == 0) return hipSuccess;
  hipLaunchKernelGGL(append_kernel, dim3((unsigned)(P.batch * P.hkv)), dim3(64), 0, s, P);
  return hipGetLastError();
}

}  // namespace fdkv
