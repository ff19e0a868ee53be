// A batch through a stack of MoE blocks (Sec. 2.1's transformer blocks with the
// attention half left out): h <- h + MoE_l(x_l) for l = 0..L-1, x_l = h or,
// with pre_norm, the RMS-normalised h (the pre-norm of the MoE blocks of the
// models the paper runs); each block the path route -> permute -> expert FFN
// -> combine, the residual added by the combine's accumulate mode (one
// rounding of h per layer). The batch's rows are gathered into a contiguous
// buffer once, run through every layer in place, and scattered back, so the
// route step sees a dense [T, H] batch.
#include "moeflow.h"
#include "common.h"

#include <algorithm>

namespace moe {
namespace {

struct StackLayout {
  size_t xb, xn, idx, w, offs, rop, por, xp, yp, inc, pws, fws, total;
  size_t pws_bytes, fws_bytes;
};

StackLayout stack_layout(int64_t T, int64_t H, int64_t F, int32_t E, int32_t k, int32_t dtype) {
  const size_t elt = dtype == MOE_BF16 ? 2 : 4;
  const int64_t P = T * k;
  StackLayout s{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + bytes, 256);
    return at;
  };
  s.xb = take((size_t)T * H * elt);
  s.xn = take((size_t)T * H * elt);
  s.idx = take((size_t)P * 4);
  s.w = take((size_t)P * 4);
  s.offs = take((size_t)(E + 1) * 4);
  s.rop = take((size_t)P * 4);
  s.por = take((size_t)P * 4);
  s.xp = take((size_t)P * H * elt);
  s.yp = take((size_t)P * H * elt);
  s.inc = take((size_t)T * 4);
  s.pws_bytes = moe_permute_workspace(T, k, E);
  s.pws = take(s.pws_bytes);
  s.fws_bytes = moe_expert_ffn_workspace(P, H, F, E, dtype);
  s.fws = take(s.fws_bytes);
  s.total = o;
  return s;
}

// dst row i = src row rows[i] (gather) or dst row rows[i] = src row i (scatter)
template <bool SCATTER>
__global__ void stack_rows_kernel(const char* __restrict__ src, char* __restrict__ dst,
                                  const int32_t* __restrict__ rows, int64_t T, int64_t n_rows,
                                  int64_t row_chunks, int32_t* __restrict__ err) {
  const int64_t total = T * row_chunks;
  for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < total;
       q += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = q / row_chunks, c = q - i * row_chunks;
    const int64_t r = rows[i];
    if (r < 0 || r >= n_rows) {
      if (c == 0) atomicExch(err, 1);
      continue;
    }
    const int64_t si = SCATTER ? i : r, di = SCATTER ? r : i;
    reinterpret_cast<uint4*>(dst)[di * row_chunks + c] =
        reinterpret_cast<const uint4*>(src)[si * row_chunks + c];
  }
}

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(uint16_t v) { return bf16_to_f32(v); }
template <typename Tv> __device__ __forceinline__ Tv from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ uint16_t from_f32<uint16_t>(float v) {
  return f32_to_bf16(v);
}

// x = h / sqrt(mean(h^2) + eps) * weight, one block per row (fp32 sum of
// squares, one rounding of each output). VEC: bf16 rows read and written 8
// values (16 bytes) at a time.
template <typename Tv, bool VEC>
__global__ void __launch_bounds__(256)
stack_rms_norm_kernel(const Tv* __restrict__ h, const Tv* __restrict__ weight, int64_t T,
                      int64_t H, float eps, Tv* __restrict__ x) {
  __shared__ float part[256 / kWave];
  const int64_t t = blockIdx.x;
  if (t >= T) return;
  const Tv* row = h + t * H;
  float ss = 0.f;
  if constexpr (VEC) {
    const uint4* r4 = reinterpret_cast<const uint4*>(row);
    for (int64_t c = threadIdx.x; c < H / 8; c += blockDim.x) {
      const uint4 u = r4[c];
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float a = bf16_to_f32((uint16_t)(w[j] & 0xffff)), b = bf16_to_f32((uint16_t)(w[j] >> 16));
        ss += a * a;
        ss += b * b;
      }
    }
  } else {
    for (int64_t c = threadIdx.x; c < H; c += blockDim.x) {
      const float v = to_f32(row[c]);
      ss += v * v;
    }
  }
  for (int o = kWave / 2; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  if ((threadIdx.x & (kWave - 1)) == 0) part[threadIdx.x / kWave] = ss;
  __syncthreads();
  float tot = 0.f;
  for (int q = 0; q < (int)(blockDim.x / kWave); ++q) tot += part[q];
  const float inv = 1.0f / sqrtf(tot / (float)H + eps);
  if constexpr (VEC) {
    const uint4* r4 = reinterpret_cast<const uint4*>(row);
    const uint4* w4 = reinterpret_cast<const uint4*>(weight);
    uint4* x4 = reinterpret_cast<uint4*>(x + t * H);
    for (int64_t c = threadIdx.x; c < H / 8; c += blockDim.x) {
      const uint4 u = r4[c];
      const uint4 g = weight ? w4[c] : make_uint4(0, 0, 0, 0);
      const uint32_t in[4] = {u.x, u.y, u.z, u.w}, gw[4] = {g.x, g.y, g.z, g.w};
      uint32_t o[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float a = bf16_to_f32((uint16_t)(in[j] & 0xffff)) * inv;
        float b = bf16_to_f32((uint16_t)(in[j] >> 16)) * inv;
        if (weight) {
          a *= bf16_to_f32((uint16_t)(gw[j] & 0xffff));
          b *= bf16_to_f32((uint16_t)(gw[j] >> 16));
        }
        o[j] = (uint32_t)f32_to_bf16(a) | ((uint32_t)f32_to_bf16(b) << 16);
      }
      x4[c] = make_uint4(o[0], o[1], o[2], o[3]);
    }
  } else {
    for (int64_t c = threadIdx.x; c < H; c += blockDim.x) {
      float v = to_f32(row[c]) * inv;
      if (weight) v *= to_f32(weight[c]);
      x[t * H + c] = from_f32<Tv>(v);
    }
  }
}

__global__ void stack_copy_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                  int64_t n) {
  for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < n;
       q += (int64_t)gridDim.x * blockDim.x)
    dst[q] = src[q];
}

}  // namespace
}  // namespace moe

extern "C" size_t moe_stack_workspace(int64_t T, int64_t H, int64_t F, int32_t E, int32_t k,
                                      int32_t dtype) {
  if (T < 1 || H < 1 || F < 1 || E < 1 || k < 1 || (dtype != MOE_BF16 && dtype != MOE_F32))
    return 0;
  return moe::stack_layout(T, H, F, E, k, dtype).total;
}

extern "C" int moe_stack_forward(void* h, int32_t dtype, int64_t n_tokens, int64_t H,
                                 const int32_t* token_ids, int64_t T, int32_t L, int32_t E,
                                 int32_t k, int64_t F, const void* const* w_router,
                                 const void* const* w_gate, const void* const* w_up,
                                 const void* const* w_down, const int32_t* slot_of_expert,
                                 int32_t S, int32_t renormalize, int32_t pre_norm,
                                 const void* const* norm_weight, float eps, void* h_trace,
                                 int32_t* idx_trace, int32_t* err, void* workspace,
                                 size_t ws_bytes, void* stream) {
  using namespace moe;
  MOE_CHECK_ARG(h && w_router && w_gate && w_up && w_down && err);
  MOE_CHECK_ARG(dtype == MOE_BF16 || dtype == MOE_F32);
  MOE_CHECK_ARG(T >= 1 && n_tokens >= T && H >= 1 && F >= 1 && L >= 1);
  MOE_CHECK_ARG(E >= 1 && E <= 256 && k >= 1 && k <= E && S >= 1);
  MOE_CHECK_ARG(slot_of_expert || S == E);
  MOE_CHECK_ARG(renormalize == 0 || renormalize == 1);
  MOE_CHECK_ARG((pre_norm == 0 && !norm_weight) || (pre_norm == 1 && eps >= 0.f));
  MOE_CHECK_ARG(token_ids || n_tokens == T);
  const size_t elt = dtype == MOE_BF16 ? 2 : 4;
  if ((H * (int64_t)elt) % 16 != 0 || (reinterpret_cast<uintptr_t>(h) & 15) ||
      (reinterpret_cast<uintptr_t>(h_trace) & 15))
    return MOE_ERR_UNSUPPORTED;                                  // 16-byte row copies
  for (int32_t l = 0; l < L; ++l)
    MOE_CHECK_ARG(w_router[l] && w_gate[l] && w_up[l] && w_down[l] &&
                  (!norm_weight || norm_weight[l]));
  if (T > 0x7fffffff) return MOE_ERR_UNSUPPORTED;
  const StackLayout lay = stack_layout(T, H, F, E, k, dtype);
  if (!workspace || ws_bytes < lay.total || (reinterpret_cast<uintptr_t>(workspace) & 255))
    return MOE_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace);
  hipStream_t st = as_stream(stream);
  const int64_t P = T * k;
  const int64_t row_chunks = H * (int64_t)elt / 16;
  const unsigned grid = (unsigned)std::min<int64_t>(ceil_div(T * row_chunks, 256),
                                                    16 * (int64_t)device_cu_count());
  void* xb = token_ids ? static_cast<void*>(ws + lay.xb) : h;
  void* const xn = ws + lay.xn;
  auto* idx = reinterpret_cast<int32_t*>(ws + lay.idx);
  auto* w = reinterpret_cast<float*>(ws + lay.w);
  auto* offs = reinterpret_cast<int32_t*>(ws + lay.offs);
  auto* rop = reinterpret_cast<int32_t*>(ws + lay.rop);
  auto* por = reinterpret_cast<int32_t*>(ws + lay.por);
  void* xp = ws + lay.xp;
  void* yp = ws + lay.yp;
  auto* inc = reinterpret_cast<int32_t*>(ws + lay.inc);

  if (token_ids) {
    stack_rows_kernel<false><<<dim3(grid), dim3(256), 0, st>>>(
        static_cast<const char*>(h), static_cast<char*>(xb), token_ids, T, n_tokens, row_chunks,
        err);
    MOE_CHECK_LAUNCH();
  }
  int rc = MOE_OK;
  for (int32_t l = 0; l < L && rc == MOE_OK; ++l) {
    const void* xin = xb;                          // the block's input
    if (pre_norm) {
      const void* wn = norm_weight ? norm_weight[l] : nullptr;
      // rows are 16-byte aligned (H * 2 a multiple of 16); the weight vector may not be
      const bool vec = dtype == MOE_BF16 && (reinterpret_cast<uintptr_t>(wn) & 15) == 0;
      if (vec)
        stack_rms_norm_kernel<uint16_t, true><<<dim3((unsigned)T), dim3(256), 0, st>>>(
            static_cast<const uint16_t*>(xb), static_cast<const uint16_t*>(wn), T, H, eps,
            static_cast<uint16_t*>(xn));
      else if (dtype == MOE_BF16)
        stack_rms_norm_kernel<uint16_t, false><<<dim3((unsigned)T), dim3(256), 0, st>>>(
            static_cast<const uint16_t*>(xb), static_cast<const uint16_t*>(wn), T, H, eps,
            static_cast<uint16_t*>(xn));
      else
        stack_rms_norm_kernel<float, false><<<dim3((unsigned)T), dim3(256), 0, st>>>(
            static_cast<const float*>(xb), static_cast<const float*>(wn), T, H, eps,
            static_cast<float*>(xn));
      MOE_CHECK_LAUNCH();
      xin = xn;
    }
    if (h_trace) {                                 // [l][0] the state, [l][1] the block's input
      char* const tr = static_cast<char*>(h_trace) + (size_t)l * 2 * T * H * elt;
      stack_copy_kernel<<<dim3(grid), dim3(256), 0, st>>>(
          static_cast<const uint4*>(xb), reinterpret_cast<uint4*>(tr), T * row_chunks);
      MOE_CHECK_LAUNCH();
      stack_copy_kernel<<<dim3(grid), dim3(256), 0, st>>>(
          static_cast<const uint4*>(xin), reinterpret_cast<uint4*>(tr + (size_t)T * H * elt),
          T * row_chunks);
      MOE_CHECK_LAUNCH();
    }
    int32_t* const idx_l = idx_trace ? idx_trace + (int64_t)l * P : idx;
    const int32_t* const slot_l = slot_of_expert ? slot_of_expert + (int64_t)l * E : nullptr;
    rc = moe_route(xin, w_router[l], dtype, T, H, E, k, nullptr, 0, renormalize, nullptr, idx_l,
                   w, stream);
    if (rc != MOE_OK) break;
    rc = moe_permute(xin, dtype, H, T, nullptr, T, idx_l, k, E, offs, rop, por, xp, ws + lay.pws,
                     lay.pws_bytes, stream);
    if (rc != MOE_OK) break;
    rc = moe_expert_ffn(xp, dtype, P, H, F, offs, E, slot_l, S, w_gate[l], w_up[l], w_down[l], yp,
                        ws + lay.fws, lay.fws_bytes, stream);
    if (rc != MOE_OK) break;
    rc = moe_combine(yp, dtype, H, P, nullptr, T, T, k, idx_l, w, rop, slot_l, E, nullptr, 1, xb,
                     inc, stream);
  }
  if (rc != MOE_OK) return rc;
  if (token_ids) {
    stack_rows_kernel<true><<<dim3(grid), dim3(256), 0, st>>>(
        static_cast<const char*>(xb), static_cast<char*>(h), token_ids, T, n_tokens, row_chunks,
        err);
    MOE_CHECK_LAUNCH();
  }
  return MOE_OK;
}
