// Exhaustive check of the device number encoders against their integer
// definitions: every fp32 bit pattern except NaN goes through
//  * e4m3_pair (the gfx950 conversion instruction on inputs clamped to
//    +-448, used by the compress kernels for FP8 caches) and f32_to_e4m3
//    (round to nearest even, saturating at 448), and
//  * cvt_bf16x2 (the conversion instruction behind every device-side bf16
//    rounding) and bf16_bits_int (round to nearest even on the bit pattern).
// Each workgroup thread takes pairs of consecutive patterns in a grid-stride
// loop and counts its mismatches; one atomic add per thread and kind.
#include "fdkv_common.h"
#include "fdkv_kernels.h"
#include "fp8.h"

namespace fdkv {

namespace {

constexpr int kCheckThreads = 256;
constexpr int kCheckBlocks = 8192;

__global__ __launch_bounds__(kCheckThreads) void check_conversions_kernel(unsigned long long* counts) {
  constexpr uint64_t kPatterns = 1ull << 32;
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x * 2;
  unsigned long long bad8 = 0, bad16 = 0;
  for (uint64_t i = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) * 2; i < kPatterns; i += stride) {
    const uint32_t u0 = (uint32_t)i, u1 = (uint32_t)i + 1u;
    const float x0 = as_f32(u0), x1 = as_f32(u1);
    const bool nan0 = (u0 & 0x7FFFFFFFu) > 0x7F800000u, nan1 = (u1 & 0x7FFFFFFFu) > 0x7F800000u;
    const uint32_t e8 = e4m3_pair(x0, x1, 0u, false);
    bad8 += (!nan0 && (e8 & 0xFFu) != f32_to_e4m3(x0)) + (!nan1 && ((e8 >> 8) & 0xFFu) != f32_to_e4m3(x1));
    const uint32_t b16 = cvt_bf16x2(x0, x1);
    bad16 += (!nan0 && (b16 & 0xFFFFu) != bf16_bits_int(x0)) + (!nan1 && (b16 >> 16) != bf16_bits_int(x1));
  }
  if (bad8) atomicAdd(&counts[0], bad8);
  if (bad16) atomicAdd(&counts[1], bad16);
}

}  // namespace

hipError_t launch_check_conversions(unsigned long long* counts, hipStream_t s) {
  hipLaunchKernelGGL(check_conversions_kernel, dim3(kCheckBlocks), dim3(kCheckThreads), 0, s, counts);
  return hipGetLastError();
}

}  // namespace fdkv
