// Measured ceilings for the roofline report: a loop of dense bf16 MFMAs with
// no memory traffic, and a streaming read. They tell what this chip reaches
// in practice (its clock under load, its memory system) beside the published
// peaks; nothing on the path calls them.
#include "moeflow.h"
#include "common.h"

#include <algorithm>

namespace moe {
namespace {

constexpr int kProbeChains = 8;      // independent accumulators per wave
constexpr int kProbeSets = 4;        // operand sets cycled so operands keep changing

// Each wave runs iters rounds of kProbeChains 32x32x16 MFMAs; operands come
// from `src` (random bf16 values), kProbeSets sets cycled per round.
__global__ void __launch_bounds__(256)
probe_mfma_kernel(const uint16_t* __restrict__ src, int64_t iters, float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  bf16x8_t a[kProbeSets], b[kProbeSets];
#pragma unroll
  for (int s = 0; s < kProbeSets; ++s) {
    a[s] = *reinterpret_cast<const bf16x8_t*>(src + (s * 2 * 64 + lane) * 8);
    b[s] = *reinterpret_cast<const bf16x8_t*>(src + ((s * 2 + 1) * 64 + lane) * 8);
  }
  f32x16_t acc[kProbeChains];
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c)
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[c][q] = 0.f;
  for (int64_t it = 0; it < iters; it += kProbeSets) {
#pragma unroll
    for (int s = 0; s < kProbeSets; ++s)
#pragma unroll
      for (int c = 0; c < kProbeChains; ++c)
        acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s], b[(s + c) % kProbeSets], acc[c], 0,
                                                         0, 0);
  }
  float v = 0.f;
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c)
#pragma unroll
    for (int q = 0; q < 16; ++q) v += acc[c][q];
  out[blockIdx.x * blockDim.x + threadIdx.x] = v;
}

__global__ void __launch_bounds__(256)
probe_read_kernel(const uint4* __restrict__ p, int64_t n, uint32_t* __restrict__ out) {
  uint32_t acc = 0;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint4 v = p[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  out[blockIdx.x * blockDim.x + threadIdx.x] = acc;
}

__global__ void __launch_bounds__(256)
probe_copy_kernel(const uint4* __restrict__ p, int64_t n, uint4* __restrict__ q) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    q[i] = p[i];
}

}  // namespace
}  // namespace moe

extern "C" int64_t moe_probe_mfma_bf16(const void* src, int64_t iters, float* out,
                                       int32_t out_len, void* stream) {
  using namespace moe;
  MOE_CHECK_ARG(src && out && iters >= 1 && iters % kProbeSets == 0);
  const int64_t blocks = 4 * (int64_t)device_cu_count();       // 4 waves per SIMD
  MOE_CHECK_ARG(out_len >= blocks * 256);
  probe_mfma_kernel<<<dim3((unsigned)blocks), dim3(256), 0, as_stream(stream)>>>(
      static_cast<const uint16_t*>(src), iters, out);
  if (hipGetLastError() != hipSuccess) return -MOE_ERR_HIP;
  // flops: blocks x 4 waves x iters x chains x (32 x 32 x 16 x 2)
  return blocks * 4 * iters * kProbeChains * 32 * 32 * 16 * 2;
}

extern "C" int moe_probe_read(const void* src, int64_t bytes, uint32_t* out, int32_t out_len,
                              void* stream) {
  using namespace moe;
  MOE_CHECK_ARG(src && out && bytes >= 16 && bytes % 16 == 0 &&
                (reinterpret_cast<uintptr_t>(src) & 15) == 0);
  const int64_t blocks = 8 * (int64_t)device_cu_count();
  MOE_CHECK_ARG(out_len >= blocks * 256);
  probe_read_kernel<<<dim3((unsigned)blocks), dim3(256), 0, as_stream(stream)>>>(
      static_cast<const uint4*>(src), bytes / 16, out);
  MOE_CHECK_LAUNCH();
  return MOE_OK;
}

extern "C" int moe_probe_copy(const void* src, void* dst, int64_t bytes, void* stream) {
  using namespace moe;
  MOE_CHECK_ARG(src && dst && bytes >= 16 && bytes % 16 == 0 &&
                (reinterpret_cast<uintptr_t>(src) & 15) == 0 &&
                (reinterpret_cast<uintptr_t>(dst) & 15) == 0);
  const int64_t blocks = 8 * (int64_t)device_cu_count();
  probe_copy_kernel<<<dim3((unsigned)blocks), dim3(256), 0, as_stream(stream)>>>(
      static_cast<const uint4*>(src), bytes / 16, static_cast<uint4*>(dst));
  MOE_CHECK_LAUNCH();
  return MOE_OK;
}
