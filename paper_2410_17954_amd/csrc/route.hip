// moe_route: router projection, top-k selection and softmax gates
// (the gating of Sec. 2.1 of the ExpertFlow paper).
//
// bf16 inputs: the projection z = x . W_g^T runs on MFMA (v_mfma_f32_16x16x32_bf16,
// float32 accumulation). A block of 4 waves owns 16 tokens; the K dimension is
// split across the 4 waves (wave w takes K-steps w, w+4, ...) so that a
// streaming read of x has many loads in flight, and the four partial sums are
// added in LDS in fixed wave order. The same block then selects the top-k of
// each token and computes its gates.
// float32 inputs (small, correctness-oriented): one block per token, one
// thread per expert.
#include "common.h"

#include <math.h>

namespace moe {
namespace {

constexpr int kRouteTok = 16;     // tokens per block (MFMA M)
constexpr int kRouteWaves = 4;

// Top-k of z[0..E) in the order (descending value, ascending index), then
// softmax gates. z may live in LDS or global memory.
__device__ void topk_softmax(const float* z, int E, int k, int renorm,
                             int32_t* __restrict__ idx_out, float* __restrict__ w_out) {
  float m = z[0];
  for (int e = 1; e < E; ++e) m = fmaxf(m, z[e]);
  float total = 0.f;
  for (int e = 0; e < E; ++e) total += expf(z[e] - m);
  float prev_v = INFINITY;
  int prev_e = -1;
  float sel = 0.f;
  for (int j = 0; j < k; ++j) {
    float bv = -INFINITY;
    int be = -1;
    for (int e = 0; e < E; ++e) {
      const float v = z[e];
      const bool after_prev = (v < prev_v) || (v == prev_v && e > prev_e);
      if (after_prev && (be < 0 || v > bv)) {
        bv = v;
        be = e;
      }
    }
    const float ev = expf(bv - m);
    idx_out[j] = be;
    w_out[j] = ev;
    sel += ev;
    prev_v = bv;
    prev_e = be;
  }
  const float den = renorm ? sel : total;
  for (int j = 0; j < k; ++j) w_out[j] = w_out[j] / den;
}

// NEB = number of 16-expert column blocks held per wave (E <= 16 * NEB).
template <int NEB>
__global__ void __launch_bounds__(256)
route_bf16_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ wg,
                  int64_t T, int64_t H, int E, int k,
                  const float* __restrict__ bias, int bias_mode, int renorm,
                  float* __restrict__ logits, int32_t* __restrict__ topk_idx,
                  float* __restrict__ topk_w) {
  constexpr int EP = NEB * 16;                    // padded expert count
  __shared__ float red[kRouteWaves][kRouteTok][EP];
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int64_t tok0 = (int64_t)blockIdx.x * kRouteTok;

  f32x4_t acc[NEB];
#pragma unroll
  for (int b = 0; b < NEB; ++b) acc[b] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int row = lane & 15;                      // token row / expert column
  const int kq = (lane >> 4) * 8;                 // this lane's 8-wide K slice
  const bool row_ok = tok0 + row < T;
  const uint16_t* xrow = x + (tok0 + row) * H + kq;
  const int64_t ksteps = (H + 31) / 32;

  constexpr int U = 4;
  for (int64_t s0 = wave; s0 < ksteps; s0 += kRouteWaves * U) {
    bf16x8_t a[U];
    bf16x8_t b[U][NEB];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t s = s0 + (int64_t)u * kRouteWaves;
      const int64_t kk = s * 32 + kq;
      const bool k_ok = (s < ksteps) && (kk < H);
      uint4 va = make_uint4(0, 0, 0, 0);
      if (k_ok && row_ok) va = *reinterpret_cast<const uint4*>(xrow + s * 32);
      a[u] = __builtin_bit_cast(bf16x8_t, va);
#pragma unroll
      for (int nb = 0; nb < NEB; ++nb) {
        const int e = nb * 16 + row;
        uint4 vb = make_uint4(0, 0, 0, 0);
        if (k_ok && e < E) vb = *reinterpret_cast<const uint4*>(wg + (int64_t)e * H + kk);
        b[u][nb] = __builtin_bit_cast(bf16x8_t, vb);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int nb = 0; nb < NEB; ++nb)
        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u], b[u][nb], acc[nb], 0, 0, 0);
  }

  // C layout of the 16x16 MFMA: lane holds column (lane % 16), rows
  // 4 * (lane / 16) + i.
#pragma unroll
  for (int nb = 0; nb < NEB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][(lane >> 4) * 4 + i][nb * 16 + row] = acc[nb][i];
  __syncthreads();

  for (int q = threadIdx.x; q < kRouteTok * EP; q += blockDim.x) {
    const int t = q / EP, e = q % EP;
    float z = ((red[0][t][e] + red[1][t][e]) + red[2][t][e]) + red[3][t][e];
    const int64_t tg = tok0 + t;
    if (e < E && tg < T) {
      if (bias_mode == 1) z += bias[e];
      else if (bias_mode == 2) z += bias[tg * E + e];
      if (logits) logits[tg * E + e] = z;
    }
    red[0][t][e] = z;
  }
  __syncthreads();

  if (threadIdx.x < kRouteTok) {
    const int t = threadIdx.x;
    const int64_t tg = tok0 + t;
    if (tg < T) topk_softmax(&red[0][t][0], E, k, renorm, topk_idx + tg * k, topk_w + tg * k);
  }
}

__global__ void __launch_bounds__(256)
route_f32_kernel(const float* __restrict__ x, const float* __restrict__ wg, int64_t T,
                 int64_t H, int E, int k, const float* __restrict__ bias, int bias_mode,
                 int renorm, float* __restrict__ logits, int32_t* __restrict__ topk_idx,
                 float* __restrict__ topk_w) {
  __shared__ float z[256];
  const int64_t t = blockIdx.x;
  const int e = threadIdx.x;
  if (e < E) {
    const float* xr = x + t * H;
    const float* wr = wg + (int64_t)e * H;
    float s = 0.f;
    for (int64_t h = 0; h < H; ++h) s = fmaf(xr[h], wr[h], s);
    if (bias_mode == 1) s += bias[e];
    else if (bias_mode == 2) s += bias[t * E + e];
    z[e] = s;
    if (logits) logits[t * E + e] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) topk_softmax(z, E, k, renorm, topk_idx + t * k, topk_w + t * k);
}

__global__ void __launch_bounds__(256)
route_logits_kernel(const float* __restrict__ logits, int64_t T, int E, int k, int renorm,
                    int32_t* __restrict__ topk_idx, float* __restrict__ topk_w) {
  const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (t >= T) return;
  topk_softmax(logits + t * E, E, k, renorm, topk_idx + t * k, topk_w + t * k);
}

}  // namespace
}  // namespace moe

extern "C" int moe_route(const void* x, const void* w_gate, int32_t dtype, int64_t T,
                         int64_t H, int32_t E, int32_t k, const float* bias,
                         int32_t bias_mode, int32_t renormalize, float* logits,
                         int32_t* topk_idx, float* topk_w, void* stream) {
  using namespace moe;
  MOE_CHECK_ARG(T >= 1 && E >= 1 && E <= 256 && k >= 1 && k <= E);
  MOE_CHECK_ARG(topk_idx && topk_w);
  MOE_CHECK_ARG(bias_mode >= 0 && bias_mode <= 2);
  MOE_CHECK_ARG((bias_mode == 0) == (bias == nullptr));
  MOE_CHECK_ARG(renormalize == 0 || renormalize == 1);
  MOE_CHECK_ARG(T <= (int64_t)1 << 40);
  hipStream_t st = as_stream(stream);
  const bool logits_in = (x == nullptr && w_gate == nullptr);
  if (logits_in) {
    MOE_CHECK_ARG(logits != nullptr && bias == nullptr);
    route_logits_kernel<<<dim3((unsigned)ceil_div(T, 256)), dim3(256), 0, st>>>(
        logits, T, E, k, renormalize, topk_idx, topk_w);
    MOE_CHECK_LAUNCH();
    return MOE_OK;
  }
  MOE_CHECK_ARG(x && w_gate && H >= 1);
  MOE_CHECK_ARG(valid_dtype(dtype));
  if (dtype == MOE_F32) {
    if (T > 0x7fffffff) return MOE_ERR_UNSUPPORTED;
    route_f32_kernel<<<dim3((unsigned)T), dim3(256), 0, st>>>(
        static_cast<const float*>(x), static_cast<const float*>(w_gate), T, H, E, k, bias,
        bias_mode, renormalize, logits, topk_idx, topk_w);
    MOE_CHECK_LAUNCH();
    return MOE_OK;
  }
  if (H % 8 != 0) return MOE_ERR_UNSUPPORTED;
  const int64_t blocks = ceil_div(T, kRouteTok);
  if (blocks > 0x7fffffff) return MOE_ERR_UNSUPPORTED;
  const int neb = (E + 15) / 16;
  const auto* xb = static_cast<const uint16_t*>(x);
  const auto* wb = static_cast<const uint16_t*>(w_gate);
#define MOE_ROUTE_LAUNCH(N)                                                               \
  route_bf16_kernel<N><<<dim3((unsigned)blocks), dim3(256), 0, st>>>(                    \
      xb, wb, T, H, E, k, bias, bias_mode, renormalize, logits, topk_idx, topk_w)
  if (neb <= 1) MOE_ROUTE_LAUNCH(1);
  else if (neb <= 2) MOE_ROUTE_LAUNCH(2);
  else if (neb <= 4) MOE_ROUTE_LAUNCH(4);
  else if (neb <= 8) MOE_ROUTE_LAUNCH(8);
  else MOE_ROUTE_LAUNCH(16);
#undef MOE_ROUTE_LAUNCH
  MOE_CHECK_LAUNCH();
  return MOE_OK;
}
