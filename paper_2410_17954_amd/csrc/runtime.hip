// Library-level helpers: status names, device query cache, fill kernels.
#include "common.h"

#include <atomic>

namespace moe {

namespace {
constexpr int kMaxDevices = 64;
std::atomic<int> g_cu_count[kMaxDevices];

__global__ void fill_i32_kernel(int32_t* __restrict__ p, int32_t v, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

__global__ void fill_i64_kernel(int64_t* __restrict__ p, int64_t v, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}
}  // namespace

int device_cu_count() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 256;
  if (dev < kMaxDevices) {
    int c = g_cu_count[dev].load(std::memory_order_relaxed);
    if (c > 0) return c;
  }
  int cu = 0;
  if (hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cu <= 0)
    cu = 256;
  if (dev < kMaxDevices) g_cu_count[dev].store(cu, std::memory_order_relaxed);
  return cu;
}

hipError_t fill_i32(int32_t* p, int32_t v, int64_t n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = ceil_div(n, 256);
  if (blocks > 1024) blocks = 1024;
  fill_i32_kernel<<<dim3((unsigned)blocks), dim3(256), 0, stream>>>(p, v, n);
  return hipGetLastError();
}

hipError_t fill_i64(int64_t* p, int64_t v, int64_t n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = ceil_div(n, 256);
  if (blocks > 1024) blocks = 1024;
  fill_i64_kernel<<<dim3((unsigned)blocks), dim3(256), 0, stream>>>(p, v, n);
  return hipGetLastError();
}

}  // namespace moe

extern "C" int moe_abi_version(void) { return MOEFLOW_ABI_VERSION; }

extern "C" const char* moe_status_str(int status) {
  switch (status) {
    case MOE_OK: return "ok";
    case MOE_ERR_ARG: return "invalid argument";
    case MOE_ERR_UNSUPPORTED: return "unsupported configuration";
    case MOE_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
    case MOE_ERR_HIP: return "HIP launch failed";
    default: return "unknown status";
  }
}
