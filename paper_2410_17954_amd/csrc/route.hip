// moe_route: router projection, top-k selection and softmax gates
// (the gating of Sec. 2.1 of the ExpertFlow paper).
//
// bf16 inputs: the projection z = x . W_g^T runs on MFMA (v_mfma_f32_16x16x32_bf16),
// in float32 chains of 8 K-steps that are added into float64 accumulators.
// Up to 32 and above 64 experts: 16 tokens per block, the K dimension split
// into contiguous ranges over the waves. 33-64 experts: 16 to 64 tokens per
// block in tiles of 16, the waves of a tile splitting the experts, the router
// matrix staged through LDS chunk by chunk. The same block then selects the top-k of each token exactly (see
// route_decide) and computes its gates.
// float32 inputs (small, correctness-oriented): one block per token, one
// thread per expert, float64 logits.
#include "common.h"

#include <math.h>

namespace moe {
namespace {

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

// ---------------------------------------------------------------- rows of 16
// Every reduction of the decision runs over a row of 16 lanes (one token per
// row, four per wave) with DPP moves: quad_perm [1,0,3,2], quad_perm
// [2,3,0,1], row_half_mirror, row_mirror. After the four steps every lane of
// the row holds the row's result.
constexpr int kRowLanes = 16;

template <int CTRL>
__device__ __forceinline__ int dpp_i32(int v) {
  return __builtin_amdgcn_mov_dpp(v, CTRL, 0xF, 0xF, true);
}
template <int CTRL>
__device__ __forceinline__ int dpp(int v) { return dpp_i32<CTRL>(v); }
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(dpp_i32<CTRL>(__float_as_int(v)));
}
template <int CTRL>
__device__ __forceinline__ double dpp(double v) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)dpp_i32<CTRL>((int)(uint32_t)b);
  const uint32_t hi = (uint32_t)dpp_i32<CTRL>((int)(uint32_t)(b >> 32));
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// Arg-max under the order (larger value first, then lower index); e < 0
// marks an empty slot.
template <int C, typename VT>
__device__ __forceinline__ void argmax_step(VT& v, int& e) {
  const VT ov = dpp<C>(v);
  const int oe = dpp<C>(e);
  if (oe >= 0 && (e < 0 || ov > v || (ov == v && oe < e))) {
    v = ov;
    e = oe;
  }
}
template <typename VT>
__device__ __forceinline__ void row_argmax(VT& v, int& e) {
  argmax_step<0xB1>(v, e);
  argmax_step<0x4E>(v, e);
  argmax_step<0x141>(v, e);
  argmax_step<0x140>(v, e);
}

// The same reductions for P independent tokens per row, step by step, so
// that the P chains of DPP moves overlap.
template <int P, typename VT>
__device__ __forceinline__ void row_argmax_multi(VT (&v)[P], int (&e)[P]) {
#pragma unroll
  for (int p = 0; p < P; ++p) argmax_step<0xB1>(v[p], e[p]);
#pragma unroll
  for (int p = 0; p < P; ++p) argmax_step<0x4E>(v[p], e[p]);
#pragma unroll
  for (int p = 0; p < P; ++p) argmax_step<0x141>(v[p], e[p]);
#pragma unroll
  for (int p = 0; p < P; ++p) argmax_step<0x140>(v[p], e[p]);
}
template <int P>
__device__ __forceinline__ void row_max_multi(float (&v)[P]) {
#pragma unroll
  for (int p = 0; p < P; ++p) v[p] = fmaxf(v[p], dpp<0xB1>(v[p]));
#pragma unroll
  for (int p = 0; p < P; ++p) v[p] = fmaxf(v[p], dpp<0x4E>(v[p]));
#pragma unroll
  for (int p = 0; p < P; ++p) v[p] = fmaxf(v[p], dpp<0x141>(v[p]));
#pragma unroll
  for (int p = 0; p < P; ++p) v[p] = fmaxf(v[p], dpp<0x140>(v[p]));
}
template <int P>
__device__ __forceinline__ void row_sum_multi(float (&v)[P]) {
#pragma unroll
  for (int p = 0; p < P; ++p) v[p] += dpp<0xB1>(v[p]);
#pragma unroll
  for (int p = 0; p < P; ++p) v[p] += dpp<0x4E>(v[p]);
#pragma unroll
  for (int p = 0; p < P; ++p) v[p] += dpp<0x141>(v[p]);
#pragma unroll
  for (int p = 0; p < P; ++p) v[p] += dpp<0x140>(v[p]);
}

// The k largest values a row holds (row lane gl, slot r <-> expert
// gl + 16 r; ok marks real entries), in the order (descending value,
// ascending index): k rounds of row arg-max; round j's winner (uniform in the
// row, e < 0 if none) goes to on_win(j, value, expert).
template <int EPL, typename VT, typename F>
__device__ __forceinline__ void row_topk(const VT (&v)[EPL], const bool (&ok)[EPL], int k, int gl,
                                         F&& on_win) {
  bool taken[EPL];
#pragma unroll
  for (int r = 0; r < EPL; ++r) taken[r] = false;
  for (int j = 0; j < k; ++j) {
    VT bv = (VT)(-INFINITY);
    int be = -1;
#pragma unroll
    for (int r = 0; r < EPL; ++r)
      if (ok[r] && !taken[r] && (be < 0 || v[r] > bv)) {
        bv = v[r];
        be = gl + kRowLanes * r;
      }
    row_argmax(bv, be);
    on_win(j, bv, be);
#pragma unroll
    for (int r = 0; r < EPL; ++r)
      if (gl + kRowLanes * r == be) taken[r] = true;
  }
}

__device__ __forceinline__ void lds_wave_sync() {
  __builtin_amdgcn_wave_barrier();
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ uint4 abs_bf16x8(uint4 v) {
  return make_uint4(v.x & 0x7fff7fffu, v.y & 0x7fff7fffu, v.z & 0x7fff7fffu, v.w & 0x7fff7fffu);
}

// K-steps (of 32) accumulated in one float32 chain before it is added to the
// float64 accumulator (the kernel for up to 32 or more than 64 experts; the
// one for 33-64 experts closes chains of one or four K-steps).
constexpr int kChainSteps = 8;

// Exactness of the decision. A logit is an exact sum of exact bf16 products
// (8-bit significands: every product is exact in float32). Each product passes
// through at most 32 * CH float32 additions (one chain of CH K-steps, whatever
// the order inside the matrix core) before the chain is added in float64, so
// |z_f32 - z| <= 2 gamma_n S + tiny with n = 32 * CH + 1 and
// S = sum_h |x_h w_eh| (the factor 2 covers directed rounding inside the
// matrix core; the float64 additions and the final rounding to float32 are the
// rest). The float32 top-k is exact, set and order, when the intervals
// [z - b, z + b] of consecutive selected experts are disjoint and every other
// expert's upper bound lies below the k-th selected lower bound. Otherwise the
// experts whose upper bound reaches the smallest selected lower bound -- a set
// that holds the exact top-k, since k experts lie above that value -- are
// recomputed in float64 (exact bf16 products, error ~1e-16 relative) and
// decide.
template <int EP>
struct DecideLds {
  float (*zf)[EP];      // float32 logits, bias included
  float (*sf)[EP];      // sum_h |x_h w_eh|
  double (*z64)[EP];    // float64 logits of refined candidates
  uint8_t (*sel)[EP];   // selected experts, in order
  float* lk;            // k-th largest lower bound per token
  int* need;            // token is decided in float64
  uint16_t* pairs;      // queued (token, expert) as t * EP + e
  int* npairs;
};

template <int EP, int TB, int NW, int CH>
__device__ __forceinline__ void route_decide(const DecideLds<EP>& s, const uint16_t* __restrict__ x,
                                             const uint16_t* __restrict__ wg, int64_t T, int64_t H,
                                             int E, int k, const float* __restrict__ bias,
                                             int bias_mode, int renorm, int64_t tok0,
                                             float* __restrict__ logits,
                                             int32_t* __restrict__ topk_idx,
                                             float* __restrict__ topk_w) {
  constexpr int EPL = EP / kRowLanes;             // expert slots per lane
  constexpr int TPP = NW * (kWave / kRowLanes);   // tokens per pass
  constexpr int P = (TB + TPP - 1) / TPP;         // passes, processed side by side
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int grp = lane / kRowLanes, gl = lane % kRowLanes;
  const float u = 5.9604645e-8f;                  // 2^-24
  const float nacc = (float)(32 * CH + 1);
  const float gam = nacc * u / (1.f - nacc * u);
  const float f64_part = (float)((H / (32 * CH) + NW + 4) * 2.3e-16);
  const float cb = 1.01f * (2.f * gam / (1.f - 2.f * gam) + f64_part);
  auto bound = [&](float z, float sabs) { return cb * sabs + 2.02f * u * fabsf(z); };

  int tt[P];
  bool live[P];
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const int t = p * TPP + wave * (kWave / kRowLanes) + grp;
    live[p] = t < TB && tok0 + t < T;
    tt[p] = t < TB ? t : 0;
  }

  // (a) float32 top-k of every token with a certificate: consecutive
  //     selected intervals disjoint and every other expert's upper bound
  //     below the k-th selected lower bound. Tokens without one queue the
  //     experts whose upper bound reaches the smallest selected lower bound
  //     (a set that holds the exact top-k) for float64 recomputation.
  {
    float z[P][EPL], bnd[P][EPL];
    bool ok[P][EPL], taken[P][EPL];
#pragma unroll
    for (int p = 0; p < P; ++p)
#pragma unroll
      for (int r = 0; r < EPL; ++r) {
        const int e = gl + kRowLanes * r;
        ok[p][r] = live[p] && e < E;
        z[p][r] = ok[p][r] ? s.zf[tt[p]][e] : 0.f;
        bnd[p][r] = ok[p][r] ? bound(z[p][r], s.sf[tt[p]][e]) : 0.f;
        taken[p][r] = false;
      }
    bool clash[P];
    float pz[P], pb[P], minlb[P];
#pragma unroll
    for (int p = 0; p < P; ++p) {
      clash[p] = false;
      pz[p] = pb[p] = 0.f;
      minlb[p] = INFINITY;
    }
    for (int j = 0; j < k; ++j) {
      float bv[P];
      int be[P];
#pragma unroll
      for (int p = 0; p < P; ++p) {
        bv[p] = -INFINITY;
        be[p] = -1;
#pragma unroll
        for (int r = 0; r < EPL; ++r)
          if (ok[p][r] && !taken[p][r] && (be[p] < 0 || z[p][r] > bv[p])) {
            bv[p] = z[p][r];
            be[p] = gl + kRowLanes * r;
          }
      }
      row_argmax_multi<P>(bv, be);
#pragma unroll
      for (int p = 0; p < P; ++p) {
        if (be[p] < 0) continue;
        const float bb = bound(bv[p], s.sf[tt[p]][be[p]]);
        if (j > 0 && fabsf(pz[p] - bv[p]) <= pb[p] + bb) clash[p] = true;
        pz[p] = bv[p];
        pb[p] = bb;
        minlb[p] = fminf(minlb[p], bv[p] - bb);
        if (live[p] && gl == 0) s.sel[tt[p]][j] = (uint8_t)be[p];
#pragma unroll
        for (int r = 0; r < EPL; ++r)
          if (gl + kRowLanes * r == be[p]) taken[p][r] = true;
      }
    }
    float ubr[P];
#pragma unroll
    for (int p = 0; p < P; ++p) {
      ubr[p] = -INFINITY;
#pragma unroll
      for (int r = 0; r < EPL; ++r)
        if (ok[p][r] && !taken[p][r]) ubr[p] = fmaxf(ubr[p], z[p][r] + bnd[p][r]);
    }
    row_max_multi<P>(ubr);
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const bool amb = clash[p] || !(ubr[p] < pz[p] - pb[p]);
      if (live[p] && gl == 0) {
        s.need[tt[p]] = amb;
        s.lk[tt[p]] = minlb[p];
      }
      if (live[p] && amb) {
#pragma unroll
        for (int r = 0; r < EPL; ++r)
          if (ok[p][r] && z[p][r] + bnd[p][r] >= minlb[p])
            s.pairs[atomicAdd(s.npairs, 1)] = (uint16_t)(tt[p] * EP + gl + kRowLanes * r);
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
  const int np = *s.npairs;
  for (int q = wave; q < np; q += NW) {
    const int t = s.pairs[q] / EP, e = s.pairs[q] % EP;
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
    for (int o = 32; o > 0; o >>= 1) a += __shfl_xor(a, o, kWave);
    if (lane == 0) s.z64[t][e] = a + (double)bias_of(bias, bias_mode, tg, E, e);
  }
  __syncthreads();

  // (c) float64 decision of the queued tokens, then the gates from the
  //     float32 logits (refined ones replaced by their float64 values rounded):
  //     softmax over all experts, restricted to the selected ones, optionally
  //     renormalised. Choice j is written by row lane j mod 16.
  float z[P][EPL];
  bool ok[P][EPL];
  bool refined[P];
  bool any_refined = false;
#pragma unroll
  for (int p = 0; p < P; ++p) {
    refined[p] = live[p] && s.need[tt[p]];
    any_refined = any_refined || ballot(refined[p]) != 0;
#pragma unroll
    for (int r = 0; r < EPL; ++r) {
      const int e = gl + kRowLanes * r;
      ok[p][r] = live[p] && e < E;
      z[p][r] = ok[p][r] ? s.zf[tt[p]][e] : 0.f;
    }
  }
  if (any_refined) {
#pragma unroll
    for (int p = 0; p < P; ++p) {
      double zd[EPL];
      bool cd[EPL];
#pragma unroll
      for (int r = 0; r < EPL; ++r) {
        const int e = gl + kRowLanes * r;
        cd[r] = refined[p] && ok[p][r] && z[p][r] + bound(z[p][r], s.sf[tt[p]][e]) >= s.lk[tt[p]];
        zd[r] = cd[r] ? s.z64[tt[p]][e] : 0.0;
        if (cd[r]) z[p][r] = (float)zd[r];
      }
      if (ballot(refined[p])) {
        row_topk<EPL>(zd, cd, k, gl, [&](int j, double, int be) {
          if (refined[p] && gl == 0 && be >= 0) s.sel[tt[p]][j] = (uint8_t)be;
        });
#pragma unroll
        for (int r = 0; r < EPL; ++r)
          if (cd[r]) s.zf[tt[p]][gl + kRowLanes * r] = z[p][r];
      }
    }
  }
  lds_wave_sync();
  float mz[P], tot[P], sp[P];
#pragma unroll
  for (int p = 0; p < P; ++p) {
    mz[p] = -INFINITY;
#pragma unroll
    for (int r = 0; r < EPL; ++r)
      if (ok[p][r]) mz[p] = fmaxf(mz[p], z[p][r]);
  }
  row_max_multi<P>(mz);
#pragma unroll
  for (int p = 0; p < P; ++p) {
    tot[p] = 0.f;
#pragma unroll
    for (int r = 0; r < EPL; ++r)
      if (ok[p][r]) tot[p] += expf(z[p][r] - mz[p]);
    sp[p] = 0.f;
    if (live[p])
      for (int j = gl; j < k; j += kRowLanes) sp[p] += expf(s.zf[tt[p]][s.sel[tt[p]][j]] - mz[p]);
  }
  row_sum_multi<P>(tot);
  row_sum_multi<P>(sp);
#pragma unroll
  for (int p = 0; p < P; ++p) {
    if (!live[p]) continue;
    const float den = renorm ? sp[p] : tot[p];
    const int64_t tg = tok0 + tt[p];
    for (int j = gl; j < k; j += kRowLanes) {
      const int e = s.sel[tt[p]][j];
      topk_idx[tg * k + j] = e;
      topk_w[tg * k + j] = expf(s.zf[tt[p]][e] - mz[p]) / den;
    }
    if (logits) {
#pragma unroll
      for (int r = 0; r < EPL; ++r)
        if (ok[p][r]) logits[tg * E + gl + kRowLanes * r] = z[p][r];
    }
  }
}

// Small or very large expert counts: 16 tokens per block, the K dimension
// split into KS contiguous ranges, one per wave (each keeps up to 8 K-steps of
// loads in flight). Partial sums are added in LDS in fixed wave order.
template <int NEB, int KS>
__global__ void __launch_bounds__(KS * 64)
route_ksplit_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ wg, int64_t T,
                    int64_t H, int E, int k, const float* __restrict__ bias, int bias_mode,
                    int renorm, float* __restrict__ logits, int32_t* __restrict__ topk_idx,
                    float* __restrict__ topk_w) {
  constexpr int EP = NEB * 16;
  constexpr int TB = 16;
  __shared__ double zacc[TB][EP];                 // also the float64 refinements afterwards
  __shared__ float sacc[TB][EP];
  __shared__ float zf[TB][EP];
  __shared__ uint8_t sel[TB][EP];
  __shared__ uint16_t pairs[TB * EP];
  __shared__ float lk[TB];
  __shared__ int need[TB];
  __shared__ int npairs;
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int64_t tok0 = (int64_t)blockIdx.x * TB;

  f32x4_t acc[NEB], acs[NEB];
  double a64[NEB][4];
#pragma unroll
  for (int b = 0; b < NEB; ++b) {
    acs[b] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < 4; ++i) a64[b][i] = 0.0;
  }
  const int row = lane & 15;                      // token row / expert column
  const int kq = (lane >> 4) * 8;                 // this lane's 8-wide K slice
  const bool row_ok = tok0 + row < T;
  const uint16_t* xrow = x + (tok0 + row) * H + kq;
  const int64_t ksteps = (H + 31) / 32;
  const int64_t spw = (ksteps + KS - 1) / KS;     // K-steps per wave, contiguous
  const int64_t s_beg = wave * spw, s_end = min(ksteps, s_beg + spw);
  constexpr int U = NEB >= 8 ? 1 : 8 / NEB;       // K-steps of loads in flight
  for (int64_t s0 = s_beg; s0 < s_end; s0 += kChainSteps) {
#pragma unroll
    for (int nb = 0; nb < NEB; ++nb) acc[nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const int64_t c_end = min(s_end, s0 + kChainSteps);
    for (int64_t s1 = s0; s1 < c_end; s1 += U) {
      uint4 a[U];
      uint4 b[U][NEB];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t s = s1 + u;
        const int64_t kk = s * 32 + kq;
        const bool k_ok = (s < c_end) && (kk < H);
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
#pragma unroll
    for (int nb = 0; nb < NEB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) a64[nb][i] += (double)acc[nb][i];
  }

  // C layout of the 16x16 MFMA: lane holds column (lane % 16), rows
  // 4 * (lane / 16) + i. Wave partials are added in wave order: all at once
  // from per-wave slots when those fit in LDS, else one wave after another.
  constexpr bool kSlots = KS * TB * EP * (sizeof(double) + sizeof(float)) <= 48 * 1024;
  if constexpr (kSlots) {
    __shared__ double zred[KS][TB][EP];
    __shared__ float sred[KS][TB][EP];
#pragma unroll
    for (int nb = 0; nb < NEB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = (lane >> 4) * 4 + i, e = nb * 16 + row;
        zred[wave][t][e] = a64[nb][i];
        sred[wave][t][e] = acs[nb][i];
      }
    __syncthreads();
    for (int q = threadIdx.x; q < TB * EP; q += blockDim.x) {
      const int t = q / EP, e = q % EP;
      double z = zred[0][t][e];
      float a = sred[0][t][e];
#pragma unroll
      for (int w = 1; w < KS; ++w) {
        z += zred[w][t][e];
        a += sred[w][t][e];
      }
      zacc[t][e] = z;
      sacc[t][e] = a;
    }
    __syncthreads();
  } else {
    for (int w = 0; w < KS; ++w) {
      if (wave == w) {
#pragma unroll
        for (int nb = 0; nb < NEB; ++nb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int t = (lane >> 4) * 4 + i, e = nb * 16 + row;
            zacc[t][e] = (w == 0 ? 0.0 : zacc[t][e]) + a64[nb][i];
            sacc[t][e] = (w == 0 ? 0.f : sacc[t][e]) + acs[nb][i];
          }
      }
      __syncthreads();
    }
  }
  for (int q = threadIdx.x; q < TB * EP; q += blockDim.x) {
    const int t = q / EP, e = q % EP;
    const int64_t tg = tok0 + t;
    double z = zacc[t][e];
    if (e < E && tg < T) z += (double)bias_of(bias, bias_mode, tg, E, e);
    zf[t][e] = (float)z;
  }
  if (threadIdx.x == 0) npairs = 0;
  __syncthreads();
  const DecideLds<EP> s{zf, sacc, zacc, sel, lk, need, pairs, &npairs};
  route_decide<EP, TB, KS, kChainSteps>(s, x, wg, T, H, E, k, bias, bias_mode, renorm, tok0,
                                        logits, topk_idx, topk_w);
}

// 33..64 experts: 64 tokens per block, one wave per 16-token tile over the
// whole K range. The router matrix is staged through LDS in chunks of
// kWChunk K-columns (one load per block instead of one per tile), the next
// chunk and the next x fragments are loaded while the current ones are used.
constexpr int kWChunk = 256;                      // K-columns per staged chunk
constexpr int kWPitch = kWChunk + 8;              // padded row (bank spread)
// 33-64 experts: blocks per compute unit wanted before a larger token tile is
// used (measured at 8192 Qwen-shaped tokens: 64-token tiles, 128 blocks, 59 us;
// 32, 256 blocks, 46 us; 16, 512 blocks, 41 us)
constexpr int kRouteTileBlocks = 2;
// float32 chain of the 33-64-expert kernel: one K-step while a wave holds one
// or two 16-expert blocks, four for four blocks (one K-step there needs more
// registers than the wave has)
constexpr int route_tile_chain(int tb) { return tb <= 32 ? 1 : 4; }

// TB tokens per block (64, 32 or 16): TB / 16 tiles of 16 tokens, the waves
// of a tile splitting the 64 expert columns between them.
template <int TB>
__global__ void __launch_bounds__(256, 2)
route_tiles_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ wg, int64_t T,
                   int64_t H, int E, int k, const float* __restrict__ bias, int bias_mode,
                   int renorm, float* __restrict__ logits, int32_t* __restrict__ topk_idx,
                   float* __restrict__ topk_w) {
  constexpr int NEB = 4, EP = 64, NW = 4;
  constexpr int TT = TB / 16;                     // 16-token tiles
  constexpr int WPT = NW / TT;                    // waves per tile
  constexpr int NEBW = NEB / WPT;                 // 16-expert blocks per wave
  static_assert(TT * WPT == NW && NEBW * WPT == NEB, "tile split");
  constexpr int SS = kWChunk / 32;                // K-steps per chunk
  constexpr int CH = route_tile_chain(TB);        // K-steps per float32 chain
  static_assert(SS % CH == 0, "whole chains per chunk");
  constexpr int WV = EP * kWChunk / 8 / (NW * kWave);   // 16-byte W pieces per thread
  __shared__ __attribute__((aligned(16))) uint16_t wsh[EP * kWPitch];   // later: z64
  __shared__ float zf[TB][EP];
  __shared__ float sf[TB][EP];
  __shared__ uint8_t sel[TB][EP];
  __shared__ uint16_t pairs[TB * EP];
  __shared__ float lk[TB];
  __shared__ int need[TB];
  __shared__ int npairs;
  static_assert(sizeof(wsh) >= sizeof(double) * TB * EP, "z64 aliases the W chunk");
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int64_t tok0 = (int64_t)blockIdx.x * TB;
  const int row = lane & 15;
  const int kq = (lane >> 4) * 8;
  const int tw = wave % TT, eg = wave / TT;       // token tile, expert group
  const bool row_ok = tok0 + tw * 16 + row < T;
  const uint16_t* xrow = x + (tok0 + tw * 16 + row) * H + kq;
  const int64_t nch = (H + kWChunk - 1) / kWChunk;

  auto load_x = [&](int64_t c, uint4 (&xa)[SS]) {
#pragma unroll
    for (int u = 0; u < SS; ++u) {
      const int64_t kk = c * kWChunk + u * 32 + kq;
      xa[u] = make_uint4(0, 0, 0, 0);
      if (row_ok && kk < H) xa[u] = *reinterpret_cast<const uint4*>(xrow + c * kWChunk + u * 32);
    }
  };
  auto load_w = [&](int64_t c, uint4 (&wr)[WV]) {
#pragma unroll
    for (int v = 0; v < WV; ++v) {
      const int q = threadIdx.x + v * NW * kWave;
      const int e = q / (kWChunk / 8), col = (q % (kWChunk / 8)) * 8;
      const int64_t kk = c * kWChunk + col;
      wr[v] = make_uint4(0, 0, 0, 0);
      if (e < E && kk < H) wr[v] = *reinterpret_cast<const uint4*>(wg + (int64_t)e * H + kk);
    }
  };
  auto store_w = [&](const uint4 (&wr)[WV]) {
#pragma unroll
    for (int v = 0; v < WV; ++v) {
      const int q = threadIdx.x + v * NW * kWave;
      const int e = q / (kWChunk / 8), col = (q % (kWChunk / 8)) * 8;
      *reinterpret_cast<uint4*>(&wsh[e * kWPitch + col]) = wr[v];
    }
  };

  f32x4_t acc[NEBW], acs[NEBW];
  double a64[NEBW][4];
#pragma unroll
  for (int b = 0; b < NEBW; ++b) {
    acs[b] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < 4; ++i) a64[b][i] = 0.0;
  }
  uint4 xc[SS], xn[SS], wr[WV];
  load_x(0, xc);
  load_w(0, wr);
  store_w(wr);
  __syncthreads();
  for (int64_t c = 0; c < nch; ++c) {
    const bool more = c + 1 < nch;
    if (more) {
      load_x(c + 1, xn);
      load_w(c + 1, wr);
    }
    // float32 chains of CH K-steps (CH MFMAs, 32 CH products) added into
    // float64: the decision's bounds are those of 32 CH + 1 float32
    // additions (8 / CH times tighter than for 8-step chains), so far fewer
    // tokens need the float64 recomputation
#pragma unroll
    for (int u = 0; u < SS; ++u) {
      const bf16x8_t av = __builtin_bit_cast(bf16x8_t, xc[u]);
      const bf16x8_t aa = __builtin_bit_cast(bf16x8_t, abs_bf16x8(xc[u]));
#pragma unroll
      for (int nb = 0; nb < NEBW; ++nb) {
        const int eb = eg * NEBW + nb;
        const uint4 bv = *reinterpret_cast<const uint4*>(&wsh[(eb * 16 + row) * kWPitch + u * 32 + kq]);
        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            av, __builtin_bit_cast(bf16x8_t, bv),
            u % CH == 0 ? f32x4_t{0.f, 0.f, 0.f, 0.f} : acc[nb], 0, 0, 0);
        acs[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            aa, __builtin_bit_cast(bf16x8_t, abs_bf16x8(bv)), acs[nb], 0, 0, 0);
      }
      if ((u + 1) % CH == 0) {
#pragma unroll
        for (int nb = 0; nb < NEBW; ++nb)
#pragma unroll
          for (int i = 0; i < 4; ++i) a64[nb][i] += (double)acc[nb][i];
      }
    }
    __syncthreads();                              // every wave is done with this chunk
    if (more) {
      store_w(wr);
#pragma unroll
      for (int u = 0; u < SS; ++u) xc[u] = xn[u];
    }
    __syncthreads();
  }

  // C layout of the 16x16 MFMA: lane holds column (lane % 16), rows
  // 4 * (lane / 16) + i of this wave's tile.
#pragma unroll
  for (int nb = 0; nb < NEBW; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = tw * 16 + (lane >> 4) * 4 + i, e = (eg * NEBW + nb) * 16 + row;
      const int64_t tg = tok0 + t;
      double z = a64[nb][i];
      if (e < E && tg < T) z += (double)bias_of(bias, bias_mode, tg, E, e);
      zf[t][e] = (float)z;
      sf[t][e] = acs[nb][i];
    }
  if (threadIdx.x == 0) npairs = 0;
  __syncthreads();
  const DecideLds<EP> s{zf, sf, reinterpret_cast<double(*)[EP]>(wsh), sel, lk, need, pairs,
                        &npairs};
  route_decide<EP, TB, NW, CH>(s, x, wg, T, H, E, k, bias, bias_mode, renorm, tok0, logits,
                               topk_idx, topk_w);
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

// Routing paths from predictor logits: row r (a token at one layer) gets the
// k experts with the largest logits, descending, equal logits lower id first.
// One thread per row; the row is scanned k times (E <= 256, k small).
__global__ void binarize_kernel(const float* __restrict__ logits, int64_t rows, int E, int k,
                                uint8_t* __restrict__ routes) {
  const int64_t r = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (r >= rows) return;
  const float* z = logits + r * E;
  float prev_v = INFINITY;
  int prev_e = -1;
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
    routes[r * k + j] = (uint8_t)(be < 0 ? 0 : be);
    prev_v = bv;
    prev_e = be;
  }
}

}  // namespace
}  // namespace moe

extern "C" int moe_route_binarize(const float* logits, int64_t rows, int32_t E, int32_t k,
                                  uint8_t* routes, void* stream) {
  using namespace moe;
  MOE_CHECK_ARG(logits && routes && rows >= 1 && E >= 1 && E <= 256 && k >= 1 && k <= E);
  if (ceil_div(rows, 256) > 0x7fffffff) return MOE_ERR_UNSUPPORTED;
  binarize_kernel<<<dim3((unsigned)ceil_div(rows, 256)), dim3(256), 0, as_stream(stream)>>>(
      logits, rows, E, k, routes);
  MOE_CHECK_LAUNCH();
  return MOE_OK;
}

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
  const int64_t blocks = ceil_div(T, 16);
  if (blocks > 0x7fffffff) return MOE_ERR_UNSUPPORTED;
  const int neb = (E + 15) / 16;
  const auto* xb = static_cast<const uint16_t*>(x);
  const auto* wb = static_cast<const uint16_t*>(w_gate);
  if (neb == 3 || neb == 4) {
    // the largest token tile that still gives every compute unit kRouteTileBlocks blocks
    const int64_t cus = device_cu_count();
    const int tb = ceil_div(T, 64) >= kRouteTileBlocks * cus ? 64
                 : ceil_div(T, 32) >= kRouteTileBlocks * cus ? 32 : 16;
    const int64_t tiles = ceil_div(T, tb);
    if (tiles > 0x7fffffff) return MOE_ERR_UNSUPPORTED;
    if (tb == 64)
      route_tiles_kernel<64><<<dim3((unsigned)tiles), dim3(256), 0, st>>>(
          xb, wb, T, H, E, k, bias, bias_mode, renormalize, logits, topk_idx, topk_w);
    else if (tb == 32)
      route_tiles_kernel<32><<<dim3((unsigned)tiles), dim3(256), 0, st>>>(
          xb, wb, T, H, E, k, bias, bias_mode, renormalize, logits, topk_idx, topk_w);
    else
      route_tiles_kernel<16><<<dim3((unsigned)tiles), dim3(256), 0, st>>>(
          xb, wb, T, H, E, k, bias, bias_mode, renormalize, logits, topk_idx, topk_w);
    MOE_CHECK_LAUNCH();
    return MOE_OK;
  }
#define MOE_ROUTE_LAUNCH(N, W)                                                            \
  route_ksplit_kernel<N, W><<<dim3((unsigned)blocks), dim3(W * 64), 0, st>>>(             \
      xb, wb, T, H, E, k, bias, bias_mode, renormalize, logits, topk_idx, topk_w)
  if (neb <= 1) MOE_ROUTE_LAUNCH(1, 8);
  else if (neb <= 2) MOE_ROUTE_LAUNCH(2, 8);
  else if (neb <= 8) MOE_ROUTE_LAUNCH(8, 4);
  else MOE_ROUTE_LAUNCH(16, 4);
#undef MOE_ROUTE_LAUNCH
  MOE_CHECK_LAUNCH();
  return MOE_OK;
}
