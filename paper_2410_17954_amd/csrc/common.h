// Shared device and host helpers of libmoeflow (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "moeflow.h"

namespace moe {

constexpr int kWave = 64;

// ---------------------------------------------------------------- bf16
// bfloat16 values travel as raw uint16 bit patterns.
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round to nearest, ties to even (NaN stays NaN): gfx950 converts in one
// branch-free instruction (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;

// ---------------------------------------------------------------- waves
__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int l = lane_id();
  return (l == 0) ? 0ull : (~0ull >> (64 - l));
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// ---------------------------------------------------------------- host
// Status helpers used by the entry points.
#define MOE_CHECK_ARG(cond) \
  do {                      \
    if (!(cond)) return MOE_ERR_ARG; \
  } while (0)

#define MOE_CHECK_LAUNCH()                              \
  do {                                                  \
    if (hipGetLastError() != hipSuccess) return MOE_ERR_HIP; \
  } while (0)

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Number of compute units of the current device (cached per device).
int device_cu_count();

// Fill `n` int32 words with `v` on `stream` (a kernel, not a memset node, so
// that the sequence stays correct inside captured HIP graphs).
hipError_t fill_i32(int32_t* p, int32_t v, int64_t n, hipStream_t stream);
hipError_t fill_i64(int64_t* p, int64_t v, int64_t n, hipStream_t stream);

inline bool valid_dtype(int32_t dt) { return dt == MOE_F32 || dt == MOE_BF16; }

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace moe
