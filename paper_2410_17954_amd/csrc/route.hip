// moe_route: router projection, top-k selection and softmax gates
// (the gating of Sec. 2.1 of the ExpertFlow paper).
//
// bf16 inputs: the projection z = x . W_g^T runs on MFMA (v_mfma_f32_16x16x32_bf16,
// float32 accumulation). A block of 4 waves owns 16 tokens; the K dimension is
// split across the 4 waves (wave w takes K-steps w, w+4, ...) so that a
// streaming read of x has many loads in flight, and the four partial sums are
// added in LDS in fixed wave order. The same block then selects the top-k of
// each token -- exactly, see route_bf16_kernel -- and computes its gates.
// float32 inputs (small, correctness-oriented): one block per token, one
// thread per expert, float64 logits.
#include "common.h"

#include <math.h>

namespace moe {
namespace {

constexpr int kRouteTok = 16;     // tokens per block (MFMA M)
constexpr int kRouteWaves = 4;

// Indices of the k largest values of v[0..E), in the order (descending value,
// ascending index). `member` (if given) restricts the candidates to a bitmask.
template <typename VT>
__device__ void select_topk(const VT* v, int E, int k, const uint64_t* member,
                            int32_t* __restrict__ idx_out) {
  VT prev_v = (VT)INFINITY;
  int prev_e = -1;
  for (int j = 0; j < k; ++j) {
    VT bv = (VT)(-INFINITY);
    int be = -1;
    for (int e = 0; e < E; ++e) {
      if (member && !((member[e >> 6] >> (e & 63)) & 1)) continue;
      const VT x = v[e];
      const bool after_prev = (x < prev_v) || (x == prev_v && e > prev_e);
      if (after_prev && (be < 0 || x > bv)) {
        bv = x;
        be = e;
      }
    }
    idx_out[j] = be;
    prev_v = bv;
    prev_e = be;
  }
}

// Softmax gates of the selected experts from float32 logits z[0..E).
__device__ void gate_weights(const float* z, int E, int k, int renorm,
                             const int32_t* __restrict__ idx, float* __restrict__ w_out) {
  float m = z[0];
  for (int e = 1; e < E; ++e) m = fmaxf(m, z[e]);
  float total = 0.f;
  for (int e = 0; e < E; ++e) total += expf(z[e] - m);
  float sel = 0.f;
  for (int j = 0; j < k; ++j) {
    const float ev = expf(z[idx[j]] - m);
    w_out[j] = ev;
    sel += ev;
  }
  const float den = renorm ? sel : total;
  for (int j = 0; j < k; ++j) w_out[j] = w_out[j] / den;
}

__device__ __forceinline__ float bias_of(const float* bias, int mode, int64_t t, int E, int e) {
  return mode == 1 ? bias[e] : (mode == 2 ? bias[t * E + e] : 0.f);
}

__device__ __forceinline__ uint4 abs_bf16x8(uint4 v) {
  return make_uint4(v.x & 0x7fff7fffu, v.y & 0x7fff7fffu, v.z & 0x7fff7fffu, v.w & 0x7fff7fffu);
}

// NEB = number of 16-expert column blocks held per wave (E <= 16 * NEB).
//
// Decisions are exact: the MFMA pass also accumulates S = sum_h |x_h w_eh|,
// which bounds the float32 error of every logit (2 gamma_{H+4} S plus the
// bias rounding; doubled to cover any accumulation order inside the matrix
// core). An expert can belong to the top-k only if its upper bound reaches
// the k-th largest lower bound. When those candidates are exactly k and their
// intervals are disjoint, the float32 order is the exact order; otherwise the
// candidates' logits are recomputed in float64 (exact bf16 products, error
// ~1e-16 relative) and the decision is taken on those.
template <int NEB>
__global__ void __launch_bounds__(256)
route_bf16_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ wg,
                  int64_t T, int64_t H, int E, int k,
                  const float* __restrict__ bias, int bias_mode, int renorm,
                  float* __restrict__ logits, int32_t* __restrict__ topk_idx,
                  float* __restrict__ topk_w) {
  constexpr int EP = NEB * 16;                    // padded expert count
  constexpr int NW = (EP + 63) / 64;              // bitmask words per token
  __shared__ __attribute__((aligned(16))) float red[kRouteWaves][kRouteTok][EP];
  __shared__ float zf[kRouteTok][EP];
  __shared__ float sf[kRouteTok][EP];
  __shared__ uint64_t umask[kRouteTok][NW];
  __shared__ int need[kRouteTok];
  __shared__ int pairs[kRouteTok * EP];           // t * EP + e
  __shared__ int npairs;
  // float64 logits of refined candidates; reuses `red` once both reductions
  // are done (16 * EP doubles <= 4 * 16 * EP floats).
  auto z64 = reinterpret_cast<double(*)[EP]>(&red[0][0][0]);
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int64_t tok0 = (int64_t)blockIdx.x * kRouteTok;

  f32x4_t acc[NEB], acs[NEB];
#pragma unroll
  for (int b = 0; b < NEB; ++b) {
    acc[b] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    acs[b] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }

  const int row = lane & 15;                      // token row / expert column
  const int kq = (lane >> 4) * 8;                 // this lane's 8-wide K slice
  const bool row_ok = tok0 + row < T;
  const uint16_t* xrow = x + (tok0 + row) * H + kq;
  const int64_t ksteps = (H + 31) / 32;

  constexpr int U = 4;
  for (int64_t s0 = wave; s0 < ksteps; s0 += kRouteWaves * U) {
    uint4 a[U];
    uint4 b[U][NEB];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t s = s0 + (int64_t)u * kRouteWaves;
      const int64_t kk = s * 32 + kq;
      const bool k_ok = (s < ksteps) && (kk < H);
      a[u] = make_uint4(0, 0, 0, 0);
      if (k_ok && row_ok) a[u] = *reinterpret_cast<const uint4*>(xrow + s * 32);
#pragma unroll
      for (int nb = 0; nb < NEB; ++nb) {
        const int e = nb * 16 + row;
        b[u][nb] = make_uint4(0, 0, 0, 0);
        if (k_ok && e < E) b[u][nb] = *reinterpret_cast<const uint4*>(wg + (int64_t)e * H + kk);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bf16x8_t av = __builtin_bit_cast(bf16x8_t, a[u]);
      const bf16x8_t aa = __builtin_bit_cast(bf16x8_t, abs_bf16x8(a[u]));
#pragma unroll
      for (int nb = 0; nb < NEB; ++nb) {
        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            av, __builtin_bit_cast(bf16x8_t, b[u][nb]), acc[nb], 0, 0, 0);
        acs[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            aa, __builtin_bit_cast(bf16x8_t, abs_bf16x8(b[u][nb])), acs[nb], 0, 0, 0);
      }
    }
  }

  // C layout of the 16x16 MFMA: lane holds column (lane % 16), rows
  // 4 * (lane / 16) + i. Sum the four K-slices in fixed wave order.
#pragma unroll
  for (int nb = 0; nb < NEB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][(lane >> 4) * 4 + i][nb * 16 + row] = acc[nb][i];
  __syncthreads();
  for (int q = threadIdx.x; q < kRouteTok * EP; q += blockDim.x) {
    const int t = q / EP, e = q % EP;
    float z = ((red[0][t][e] + red[1][t][e]) + red[2][t][e]) + red[3][t][e];
    const int64_t tg = tok0 + t;
    if (e < E && tg < T) z += bias_of(bias, bias_mode, tg, E, e);
    zf[t][e] = z;
  }
  __syncthreads();
#pragma unroll
  for (int nb = 0; nb < NEB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][(lane >> 4) * 4 + i][nb * 16 + row] = acs[nb][i];
  if (threadIdx.x == 0) npairs = 0;
  __syncthreads();
  for (int q = threadIdx.x; q < kRouteTok * EP; q += blockDim.x) {
    const int t = q / EP, e = q % EP;
    sf[t][e] = ((red[0][t][e] + red[1][t][e]) + red[2][t][e]) + red[3][t][e];
  }
  __syncthreads();

  // Candidate analysis, one thread per token.
  if (threadIdx.x < kRouteTok) {
    const int t = threadIdx.x;
    const int64_t tg = tok0 + t;
    if (tg < T) {
      const float u = 5.9604645e-8f;                       // 2^-24
      const float n = (float)(H + 4);
      const float gam = n * u / (1.f - n * u);
      const float c = 1.01f * 2.f * gam / (1.f - 2.f * gam);
      // k-th largest lower bound
      float lk = -INFINITY;
      {
        float prev = INFINITY;
        int prev_e = -1;
        for (int j = 0; j < k; ++j) {
          float bv = -INFINITY;
          int be = -1;
          for (int e = 0; e < E; ++e) {
            const float lb = zf[t][e] - (c * sf[t][e] + 2.02f * u * fabsf(zf[t][e]));
            const bool after = (lb < prev) || (lb == prev && e > prev_e);
            if (after && (be < 0 || lb > bv)) {
              bv = lb;
              be = e;
            }
          }
          prev = bv;
          prev_e = be;
          lk = bv;
        }
      }
      int cnt = 0;
      for (int w = 0; w < NW; ++w) umask[t][w] = 0;
      for (int e = 0; e < E; ++e) {
        const float ub = zf[t][e] + (c * sf[t][e] + 2.02f * u * fabsf(zf[t][e]));
        if (ub >= lk) {
          umask[t][e >> 6] |= 1ull << (e & 63);
          ++cnt;
        }
      }
      int amb = cnt > k;
      for (int e = 0; e < E && !amb; ++e) {
        if (!((umask[t][e >> 6] >> (e & 63)) & 1)) continue;
        const float be = c * sf[t][e] + 2.02f * u * fabsf(zf[t][e]);
        for (int f = e + 1; f < E; ++f) {
          if (!((umask[t][f >> 6] >> (f & 63)) & 1)) continue;
          const float bf = c * sf[t][f] + 2.02f * u * fabsf(zf[t][f]);
          if (fabsf(zf[t][e] - zf[t][f]) <= be + bf) {
            amb = 1;
            break;
          }
        }
      }
      need[t] = amb;
      if (amb)
        for (int e = 0; e < E; ++e)
          if ((umask[t][e >> 6] >> (e & 63)) & 1) {
            pairs[atomicAdd(&npairs, 1)] = t * EP + e;
          }
    } else {
      need[t] = 0;
    }
  }
  __syncthreads();

  // Float64 recomputation of the ambiguous candidates, one wave per (token,
  // expert): lanes take 8-element slices, then a fixed-order tree sum.
  for (int p = wave; p < npairs; p += kRouteWaves) {
    const int t = pairs[p] / EP, e = pairs[p] % EP;
    const int64_t tg = tok0 + t;
    const uint16_t* xr = x + tg * H;
    const uint16_t* wr = wg + (int64_t)e * H;
    double s = 0.0;
    for (int64_t h = (int64_t)lane * 8; h < H; h += kWave * 8) {
      const uint4 xv = *reinterpret_cast<const uint4*>(xr + h);
      const uint4 wv = *reinterpret_cast<const uint4*>(wr + h);
      const uint32_t xs[4] = {xv.x, xv.y, xv.z, xv.w};
      const uint32_t ws[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        s = fma((double)__uint_as_float(xs[q] << 16), (double)__uint_as_float(ws[q] << 16), s);
        s = fma((double)__uint_as_float(xs[q] & 0xffff0000u),
                (double)__uint_as_float(ws[q] & 0xffff0000u), s);
      }
    }
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, kWave);
    if (lane == 0) z64[t][e] = s + (double)bias_of(bias, bias_mode, tg, E, e);
  }
  __syncthreads();

  if (threadIdx.x < kRouteTok) {
    const int t = threadIdx.x;
    const int64_t tg = tok0 + t;
    if (tg < T) {
      int32_t* io = topk_idx + tg * k;
      if (need[t]) {
        select_topk<double>(&z64[t][0], E, k, &umask[t][0], io);
        for (int e = 0; e < E; ++e)
          if ((umask[t][e >> 6] >> (e & 63)) & 1) zf[t][e] = (float)z64[t][e];
      } else {
        select_topk<float>(&zf[t][0], E, k, nullptr, io);
      }
      gate_weights(&zf[t][0], E, k, renorm, io, topk_w + tg * k);
      if (logits)
        for (int e = 0; e < E; ++e) logits[tg * E + e] = zf[t][e];
    }
  }
}

// float32 inputs: logits in float64 (products of two floats are exact in
// float64), decision on those, gates from their float32 rounding.
__global__ void __launch_bounds__(256)
route_f32_kernel(const float* __restrict__ x, const float* __restrict__ wg, int64_t T,
                 int64_t H, int E, int k, const float* __restrict__ bias, int bias_mode,
                 int renorm, float* __restrict__ logits, int32_t* __restrict__ topk_idx,
                 float* __restrict__ topk_w) {
  __shared__ double z64[256];
  __shared__ float z[256];
  const int64_t t = blockIdx.x;
  const int e = threadIdx.x;
  if (e < E) {
    const float* xr = x + t * H;
    const float* wr = wg + (int64_t)e * H;
    double s = 0.0;
    for (int64_t h = 0; h < H; ++h) s = fma((double)xr[h], (double)wr[h], s);
    s += (double)bias_of(bias, bias_mode, t, E, e);
    z64[e] = s;
    z[e] = (float)s;
    if (logits) logits[t * E + e] = (float)s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    select_topk<double>(z64, E, k, nullptr, topk_idx + t * k);
    gate_weights(z, E, k, renorm, topk_idx + t * k, topk_w + t * k);
  }
}

__global__ void __launch_bounds__(256)
route_logits_kernel(const float* __restrict__ logits, int64_t T, int E, int k, int renorm,
                    int32_t* __restrict__ topk_idx, float* __restrict__ topk_w) {
  const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (t >= T) return;
  select_topk<float>(logits + t * E, E, k, nullptr, topk_idx + t * k);
  gate_weights(logits + t * E, E, k, renorm, topk_idx + t * k, topk_w + t * k);
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
