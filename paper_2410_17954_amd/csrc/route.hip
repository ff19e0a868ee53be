// moe_route: router projection, top-k selection and softmax gates
// (the gating of Sec. 2.1 of the ExpertFlow paper).
//
// bf16 inputs: the projection z = x . W_g^T runs on MFMA (v_mfma_f32_16x16x32_bf16,
// float32 accumulation). A block of W waves (8 for up to 64 experts, else 4)
// owns 16 tokens; the K dimension is split across the waves (wave w takes
// K-steps w, w+W, ...), each wave keeping 8 K-steps of loads in flight, so a
// streaming read of x has many loads outstanding, and the W partial sums are
// added in LDS in fixed wave order. The same block then selects the top-k of
// each token -- exactly, see route_bf16_kernel -- and computes its gates.
// float32 inputs (small, correctness-oriented): one block per token, one
// thread per expert, float64 logits.
#include "common.h"

#include <math.h>

namespace moe {
namespace {

constexpr int kRouteTok = 16;     // tokens per block (MFMA M)

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

// Reductions over groups of LPT consecutive lanes (LPT a power of two <= 64):
// xor partners stay inside a group.
// Arg-max under the order (larger value first, then lower index); e < 0
// marks an empty slot. Every lane of the group ends with the group's winner.
template <int LPT, typename VT>
__device__ __forceinline__ void grp_argmax(VT& v, int& e) {
#pragma unroll
  for (int o = LPT / 2; o > 0; o >>= 1) {
    const VT ov = __shfl_xor(v, o, kWave);
    const int oe = __shfl_xor(e, o, kWave);
    if (oe >= 0 && (e < 0 || ov > v || (ov == v && oe < e))) {
      v = ov;
      e = oe;
    }
  }
}

template <int LPT, typename VT>
__device__ __forceinline__ VT grp_max(VT v) {
#pragma unroll
  for (int o = LPT / 2; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, kWave));
  return v;
}

template <int LPT, typename VT>
__device__ __forceinline__ VT grp_sum(VT v) {
#pragma unroll
  for (int o = LPT / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// The k largest values a group holds (group lane gl, slot r <-> expert
// gl + LPT r; ok marks real entries), in the order (descending value,
// ascending index): k rounds of group arg-max. Group lane 0 writes the
// experts to sel[0..k); returns the k-th value.
template <int LPT, int EPL, typename VT>
__device__ VT grp_topk(const VT (&v)[EPL], const bool (&ok)[EPL], int k, int gl, int32_t* sel) {
  bool taken[EPL];
#pragma unroll
  for (int r = 0; r < EPL; ++r) taken[r] = false;
  VT kth = (VT)(-INFINITY);
  for (int j = 0; j < k; ++j) {
    VT bv = (VT)(-INFINITY);
    int be = -1;
#pragma unroll
    for (int r = 0; r < EPL; ++r)
      if (ok[r] && !taken[r] && (be < 0 || v[r] > bv)) {
        bv = v[r];
        be = gl + LPT * r;
      }
    grp_argmax<LPT>(bv, be);
    if (gl == 0 && sel) sel[j] = be;
    kth = bv;
#pragma unroll
    for (int r = 0; r < EPL; ++r)
      if (gl + LPT * r == be) taken[r] = true;
  }
  return kth;
}

__device__ __forceinline__ void lds_wave_sync() {
  __builtin_amdgcn_wave_barrier();
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ uint4 abs_bf16x8(uint4 v) {
  return make_uint4(v.x & 0x7fff7fffu, v.y & 0x7fff7fffu, v.z & 0x7fff7fffu, v.w & 0x7fff7fffu);
}

// NEB = number of 16-expert column blocks held per wave (E <= 16 * NEB).
//
// Decisions are exact: the MFMA pass also accumulates S = sum_h |x_h w_eh|,
// which bounds the float32 error of every logit (2 gamma_{H+W} S plus the
// bias rounding; doubled to cover any accumulation order inside the matrix
// core). An expert can belong to the top-k only if its upper bound reaches
// the k-th largest lower bound. When those candidates are exactly k and their
// intervals are disjoint, the float32 order is the exact order; otherwise the
// candidates' logits are recomputed in float64 (exact bf16 products, error
// ~1e-16 relative) and the decision is taken on those.
template <int NEB, int kRouteWaves>
__global__ void __launch_bounds__(kRouteWaves * 64)
route_bf16_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ wg,
                  int64_t T, int64_t H, int E, int k,
                  const float* __restrict__ bias, int bias_mode, int renorm,
                  float* __restrict__ logits, int32_t* __restrict__ topk_idx,
                  float* __restrict__ topk_w) {
  constexpr int EP = NEB * 16;                    // padded expert count
  constexpr int EPL = EP <= 64 ? 1 : EP / 64;     // expert slots per lane in the decision
  __shared__ __attribute__((aligned(16))) float red[kRouteWaves][kRouteTok][EP];
  __shared__ float zf[kRouteTok][EP];
  __shared__ float sf[kRouteTok][EP];
  __shared__ int32_t sel[kRouteTok][EP];          // selected experts, in order
  __shared__ int32_t pairs[kRouteTok * EP];       // (t, e) candidates to refine: t * EP + e
  __shared__ int npairs;
  __shared__ int need[kRouteTok];
  __shared__ bool queued[kRouteTok][EP];          // (t, e) is in pairs
  // float64 logits of refined candidates; reuses `red` once both reductions
  // are done (16 * EP doubles <= W * 16 * EP floats).
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

  constexpr int U = NEB >= 8 ? 1 : 8 / NEB;       // K-steps of loads in flight per wave
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
    float z = red[0][t][e];
#pragma unroll
    for (int w = 1; w < kRouteWaves; ++w) z += red[w][t][e];
    const int64_t tg = tok0 + t;
    if (e < E && tg < T) z += bias_of(bias, bias_mode, tg, E, e);
    zf[t][e] = z;
  }
  __syncthreads();
#pragma unroll
  for (int nb = 0; nb < NEB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][(lane >> 4) * 4 + i][nb * 16 + row] = acs[nb][i];
  __syncthreads();
  for (int q = threadIdx.x; q < kRouteTok * EP; q += blockDim.x) {
    const int t = q / EP, e = q % EP;
    float a = red[0][t][e];
#pragma unroll
    for (int w = 1; w < kRouteWaves; ++w) a += red[w][t][e];
    sf[t][e] = a;
  }
  if (threadIdx.x == 0) npairs = 0;
  __syncthreads();

  // Decision. Each token gets a group of LPT lanes (all EP expert slots
  // when EP <= 64, else 64 lanes with EPL slots each); a wave holds TPW
  // tokens at once, so the group reductions of several tokens overlap.
  constexpr int LPT = EP <= 64 ? EP : 64;
  constexpr int TPW = kWave / LPT;
  constexpr int PASSES = (kRouteTok + kRouteWaves * TPW - 1) / (kRouteWaves * TPW);
  const int grp = lane / LPT, gl = lane % LPT;
  const uint64_t gmask = (LPT == 64) ? ~0ull : (((1ull << LPT) - 1) << (grp * LPT));
  const float u = 5.9604645e-8f;                         // 2^-24
  const float nacc = (float)(H + kRouteWaves);            // products + wave partial sums
  const float gam = nacc * u / (1.f - nacc * u);
  const float cb = 1.01f * 2.f * gam / (1.f - 2.f * gam);

  // (a) candidates; unambiguous tokens are decided in float32, the others
  //     queue their candidates for float64 recomputation.
  for (int pass = 0; pass < PASSES; ++pass) {
    const int t = (pass * kRouteWaves + wave) * TPW + grp;
    const bool live = t < kRouteTok && tok0 + t < T;
    const int tt = t < kRouteTok ? t : 0;
    float z[EPL], bnd[EPL], lb[EPL];
    bool ok[EPL];
#pragma unroll
    for (int r = 0; r < EPL; ++r) {
      const int e = gl + LPT * r;
      ok[r] = live && e < E;
      z[r] = ok[r] ? zf[tt][e] : 0.f;
      bnd[r] = ok[r] ? cb * sf[tt][e] + 2.02f * u * fabsf(z[r]) : 0.f;
      lb[r] = z[r] - bnd[r];
    }
    const float lk = grp_topk<LPT, EPL>(lb, ok, k, gl, (int32_t*)nullptr);
    bool cand[EPL];
    int cnt = 0;
#pragma unroll
    for (int r = 0; r < EPL; ++r) {
      cand[r] = ok[r] && z[r] + bnd[r] >= lk;
      cnt += __popcll(ballot(cand[r]) & gmask);
    }
    bool amb = cnt > k;
    // Exactly k candidates: the float32 order is exact unless two intervals meet.
    bool clash = false;
#pragma unroll
    for (int rr = 0; rr < EPL; ++rr) {
      uint64_t mm = ballot(cand[rr]) & gmask;
      for (int c = 0; c < k; ++c) {            // the group's candidates, one per round
        const int l = mm ? __builtin_ctzll(mm) : lane;
        mm &= mm ? mm - 1 : 0;
        const float zc = __shfl(z[rr], l, kWave), bc = __shfl(bnd[rr], l, kWave);
#pragma unroll
        for (int r = 0; r < EPL; ++r)
          if (cand[r] && (r != rr || lane != l) && fabsf(z[r] - zc) <= bnd[r] + bc) clash = true;
      }
    }
    amb = amb || (ballot(clash) & gmask) != 0;
    grp_topk<LPT, EPL>(z, ok, k, gl, live && !amb ? sel[tt] : (int32_t*)nullptr);
    if (live && gl == 0) need[tt] = amb;
    if (live) {
#pragma unroll
      for (int r = 0; r < EPL; ++r) {
        const int e = gl + LPT * r;
        if (e < EP) queued[tt][e] = amb && cand[r];
        if (amb && cand[r]) pairs[atomicAdd(&npairs, 1)] = tt * EP + e;
      }
    }
  }
  __syncthreads();

  // (b) float64 logits of the queued candidates (bf16 products are exact in
  //     float64), one wave per candidate, four 512-element slices per round
  //     with every load issued before the FMAs; fixed-order tree sum.
  auto dot8 = [](const uint4& xv, const uint4& wv, double& a) {
    const uint32_t xs[4] = {xv.x, xv.y, xv.z, xv.w};
    const uint32_t ws[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      a = fma((double)__uint_as_float(xs[i] << 16), (double)__uint_as_float(ws[i] << 16), a);
      a = fma((double)__uint_as_float(xs[i] & 0xffff0000u),
              (double)__uint_as_float(ws[i] & 0xffff0000u), a);
    }
  };
  for (int p = wave; p < npairs; p += kRouteWaves) {
    const int t = pairs[p] / EP, e = pairs[p] % EP;
    const int64_t tg = tok0 + t;
    const uint16_t* xr = x + tg * H;
    const uint16_t* wr = wg + (int64_t)e * H;
    double a = 0.0;
    constexpr int R = 4;
    int64_t h = (int64_t)lane * 8;
    for (; h + (R - 1) * kWave * 8 < H; h += R * kWave * 8) {
      uint4 xv[R], wv[R];
#pragma unroll
      for (int i = 0; i < R; ++i) {
        xv[i] = *reinterpret_cast<const uint4*>(xr + h + i * kWave * 8);
        wv[i] = *reinterpret_cast<const uint4*>(wr + h + i * kWave * 8);
      }
#pragma unroll
      for (int i = 0; i < R; ++i) dot8(xv[i], wv[i], a);
    }
    for (; h < H; h += kWave * 8)
      dot8(*reinterpret_cast<const uint4*>(xr + h), *reinterpret_cast<const uint4*>(wr + h), a);
    const double sum = grp_sum<64>(a);
    if (lane == 0) z64[t][e] = sum + (double)bias_of(bias, bias_mode, tg, E, e);
  }
  __syncthreads();

  // (c) float64 decision of the queued tokens, then the gates from the
  //     float32 logits: softmax over all experts, restricted to the selected
  //     ones, optionally renormalised. Choice j is handled by group lane j.
  for (int pass = 0; pass < PASSES; ++pass) {
    const int t = (pass * kRouteWaves + wave) * TPW + grp;
    const bool live = t < kRouteTok && tok0 + t < T;
    const int tt = t < kRouteTok ? t : 0;
    const bool refined = live && need[tt];
    float z[EPL];
    bool ok[EPL];
#pragma unroll
    for (int r = 0; r < EPL; ++r) {
      const int e = gl + LPT * r;
      ok[r] = live && e < E;
      z[r] = ok[r] ? zf[tt][e] : 0.f;
    }
    double zd[EPL];
    bool cd[EPL];
#pragma unroll
    for (int r = 0; r < EPL; ++r) {
      const int e = gl + LPT * r;
      cd[r] = refined && ok[r] && queued[tt][e];
      zd[r] = cd[r] ? z64[tt][e] : 0.0;
      if (cd[r]) z[r] = (float)zd[r];
    }
    grp_topk<LPT, EPL>(zd, cd, k, gl, refined ? sel[tt] : (int32_t*)nullptr);
#pragma unroll
    for (int r = 0; r < EPL; ++r)
      if (ok[r]) zf[tt][gl + LPT * r] = z[r];
    lds_wave_sync();
    float mz = -INFINITY;
#pragma unroll
    for (int r = 0; r < EPL; ++r)
      if (ok[r]) mz = fmaxf(mz, z[r]);
    mz = grp_max<LPT>(mz);
    float part = 0.f;
#pragma unroll
    for (int r = 0; r < EPL; ++r)
      if (ok[r]) part += expf(z[r] - mz);
    const float total = grp_sum<LPT>(part);
    float selpart = 0.f;
    if (live)
      for (int j = gl; j < k; j += LPT) selpart += expf(zf[tt][sel[tt][j]] - mz);
    const float den = renorm ? grp_sum<LPT>(selpart) : total;
    if (live) {
      const int64_t tg = tok0 + tt;
      for (int j = gl; j < k; j += LPT) {
        const int e = sel[tt][j];
        topk_idx[tg * k + j] = e;
        topk_w[tg * k + j] = expf(zf[tt][e] - mz) / den;
      }
      if (logits) {
#pragma unroll
        for (int r = 0; r < EPL; ++r)
          if (ok[r]) logits[tg * E + gl + LPT * r] = z[r];
      }
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
#define MOE_ROUTE_LAUNCH(N, W)                                                            \
  route_bf16_kernel<N, W><<<dim3((unsigned)blocks), dim3(W * 64), 0, st>>>(               \
      xb, wb, T, H, E, k, bias, bias_mode, renormalize, logits, topk_idx, topk_w)
  if (neb <= 1) MOE_ROUTE_LAUNCH(1, 8);
  else if (neb <= 2) MOE_ROUTE_LAUNCH(2, 8);
  else if (neb <= 4) MOE_ROUTE_LAUNCH(4, 8);
  else if (neb <= 8) MOE_ROUTE_LAUNCH(8, 4);
  else MOE_ROUTE_LAUNCH(16, 4);
#undef MOE_ROUTE_LAUNCH
  MOE_CHECK_LAUNCH();
  return MOE_OK;
}
