// moe_combine: gate-weighted sum of expert outputs per token (Sec. 2.1), over
// experts resident in the expert cache, plus always-on shared experts.
//
// One wavefront per batch token; each lane owns 8 consecutive features at a
// time (16-byte bf16 vectors) and accumulates in float32 in ascending choice
// order, adds the shared-expert row and, in accumulate mode, the existing
// output, and rounds once.
// bf16 with k <= 8 (combine_bf16_kernel): lane j loads choice j's row index
// first, so the loads of the rows start while the token -> expert -> slot
// chain that decides residency is still in flight (rows of missed experts
// are read but not used); each round issues 8 row loads per lane (k choices x
// 8/k feature groups) before accumulating. Other cases (combine_kernel) stage
// the choices in LDS and walk the features one group at a time.
#include "common.h"

namespace moe {
namespace {

constexpr int kCombWaves = 4;

struct CombArgs {
  const void* y_perm;
  int64_t H, rows;
  const int32_t* token_ids;
  int64_t T, n_tokens;
  int k;
  const int32_t* idx;
  const float* w;
  const int32_t* row_of_pair;
  const int32_t* slot;
  int E;
  const void* y_shared;
  int accumulate;
  void* y;
  int32_t* incomplete;
};

template <bool BF16>
__device__ __forceinline__ void load8(const void* base, int64_t off, float v[8]) {
  if (BF16) {
    const uint4 q = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + off);
    const uint32_t u[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(u[i] << 16);
      v[2 * i + 1] = __uint_as_float(u[i] & 0xffff0000u);
    }
  } else {
    const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(base) + off);
    const float4 a = p[0], b = p[1];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
}

template <bool BF16>
__device__ __forceinline__ void store8(void* base, int64_t off, const float v[8]) {
  if (BF16) {
    uint32_t u[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      u[i] = (uint32_t)f32_to_bf16(v[2 * i]) | ((uint32_t)f32_to_bf16(v[2 * i + 1]) << 16);
    *reinterpret_cast<uint4*>(static_cast<uint16_t*>(base) + off) = make_uint4(u[0], u[1], u[2], u[3]);
  } else {
    float4* p = reinterpret_cast<float4*>(static_cast<float*>(base) + off);
    p[0] = make_float4(v[0], v[1], v[2], v[3]);
    p[1] = make_float4(v[4], v[5], v[6], v[7]);
  }
}

// Features are processed 8 at a time; f32 rows need H % 4 == 0, so a last
// group of 4 is handled by the scalar tail below.
template <bool BF16>
__global__ void __launch_bounds__(kCombWaves * kWave)
combine_kernel(CombArgs a) {
  __shared__ int32_t s_row[kCombWaves][256];
  __shared__ float s_w[kCombWaves][256];
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  const int64_t i = (int64_t)blockIdx.x * kCombWaves + wave;
  int64_t t = -1;
  if (i < a.T) {
    t = a.token_ids ? (int64_t)a.token_ids[i] : i;
    if (t >= a.n_tokens) t = -1;
  }
  const bool active = t >= 0;
  int missing = 0;
  if (active) {
    for (int j = lane; j < a.k; j += kWave) {
      const int e = a.idx[t * a.k + j];
      bool resident = true;
      if (a.slot) resident = (e >= 0 && e < a.E) && a.slot[e] >= 0;
      const int32_t r = a.row_of_pair[i * a.k + j];
      const bool ok = resident && r >= 0 && r < a.rows;
      s_row[wave][j] = ok ? r : -1;
      s_w[wave][j] = a.w[t * a.k + j];
      if (!resident) missing = 1;
    }
  }
  missing = __any(missing);
  if (active && lane == 0 && a.incomplete) a.incomplete[i] = missing;
  __syncthreads();
  if (!active) return;

  const int64_t H = a.H;
  const int64_t groups = H / 8;
  for (int64_t g = lane; g < groups; g += kWave) {
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < a.k; ++j) {
      const int32_t r = s_row[wave][j];
      if (r < 0) continue;
      const float wj = s_w[wave][j];
      float v[8];
      load8<BF16>(a.y_perm, (int64_t)r * H + g * 8, v);
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[q] = fmaf(wj, v[q], acc[q]);
    }
    if (a.y_shared) {
      float v[8];
      load8<BF16>(a.y_shared, i * H + g * 8, v);
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[q] += v[q];
    }
    if (a.accumulate) {
      float v[8];
      load8<BF16>(a.y, t * H + g * 8, v);
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[q] += v[q];
    }
    store8<BF16>(a.y, t * H + g * 8, acc);
  }
  if (!BF16) {
    // f32 tail of 4 features when H % 8 == 4.
    const int64_t h0 = groups * 8;
    for (int64_t h = h0 + lane; h < H; h += kWave) {
      float acc = 0.f;
      for (int j = 0; j < a.k; ++j) {
        const int32_t r = s_row[wave][j];
        if (r < 0) continue;
        acc = fmaf(s_w[wave][j], static_cast<const float*>(a.y_perm)[(int64_t)r * H + h], acc);
      }
      if (a.y_shared) acc += static_cast<const float*>(a.y_shared)[i * H + h];
      if (a.accumulate) acc += static_cast<float*>(a.y)[t * H + h];
      static_cast<float*>(a.y)[t * H + h] = acc;
    }
  }
}

template <int KB>
__global__ void __launch_bounds__(kCombWaves * kWave)
combine_bf16_kernel(CombArgs a) {
  constexpr int CU = 8 / KB;                      // feature groups per round
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  const int64_t i = (int64_t)blockIdx.x * kCombWaves + wave;
  if (i >= a.T) return;                           // whole wave
  const int k = a.k;
  const int32_t r_l = lane < k ? a.row_of_pair[i * k + lane] : -1;
  int64_t t = a.token_ids ? (int64_t)a.token_ids[i] : i;
  const bool active = t >= 0 && t < a.n_tokens;
  if (!active) t = 0;
  int e_l = -1;
  float w_l = 0.f;
  bool res_l = false;
  if (active && lane < k) {
    e_l = a.idx[t * k + lane];
    w_l = a.w[t * k + lane];
    res_l = a.slot ? (e_l >= 0 && e_l < a.E && a.slot[e_l] >= 0) : true;
  }
  const bool ok_l = res_l && r_l >= 0 && r_l < a.rows;
  const bool missing = ballot(active && lane < k && !res_l) != 0;
  if (active && lane == 0 && a.incomplete) a.incomplete[i] = missing ? 1 : 0;
  if (!active) return;
  int32_t rj[KB];
  float wj[KB];
  bool okj[KB];
#pragma unroll
  for (int j = 0; j < KB; ++j) {
    rj[j] = __shfl(r_l, j, kWave);
    wj[j] = __shfl(w_l, j, kWave);
    okj[j] = j < k && __shfl(ok_l ? 1 : 0, j, kWave) != 0;
    if (!(j < k && rj[j] >= 0 && rj[j] < a.rows)) rj[j] = -1;
  }
  const int64_t H = a.H, G = H / 8;
  const uint16_t* yp = static_cast<const uint16_t*>(a.y_perm);
  for (int64_t g0 = 0; g0 < G; g0 += (int64_t)kWave * CU) {
    uint4 v[KB][CU];
#pragma unroll
    for (int j = 0; j < KB; ++j)
#pragma unroll
      for (int c = 0; c < CU; ++c) {
        const int64_t g = g0 + c * kWave + lane;
        v[j][c] = (rj[j] >= 0 && g < G) ? *reinterpret_cast<const uint4*>(yp + (int64_t)rj[j] * H + g * 8)
                                        : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
    for (int c = 0; c < CU; ++c) {
      const int64_t g = g0 + c * kWave + lane;
      if (g >= G) continue;
      float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < KB; ++j) {
        if (!okj[j]) continue;
        const uint32_t u[4] = {v[j][c].x, v[j][c].y, v[j][c].z, v[j][c].w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[2 * q] = fmaf(wj[j], __uint_as_float(u[q] << 16), acc[2 * q]);
          acc[2 * q + 1] = fmaf(wj[j], __uint_as_float(u[q] & 0xffff0000u), acc[2 * q + 1]);
        }
      }
      if (a.y_shared) {
        float sv[8];
        load8<true>(a.y_shared, i * H + g * 8, sv);
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[q] += sv[q];
      }
      if (a.accumulate) {
        float yv[8];
        load8<true>(a.y, t * H + g * 8, yv);
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[q] += yv[q];
      }
      store8<true>(a.y, t * H + g * 8, acc);
    }
  }
}

}  // namespace
}  // namespace moe

extern "C" int moe_combine(const void* y_perm, int32_t dtype, int64_t H, int64_t rows,
                           const int32_t* token_ids, int64_t T, int64_t n_tokens, int32_t k,
                           const int32_t* topk_idx, const float* topk_w,
                           const int32_t* row_of_pair, const int32_t* slot_of_expert,
                           int32_t E, const void* y_shared, int32_t accumulate, void* y,
                           int32_t* incomplete, void* stream) {
  using namespace moe;
  MOE_CHECK_ARG(y_perm && topk_idx && topk_w && row_of_pair && y);
  MOE_CHECK_ARG(valid_dtype(dtype));
  MOE_CHECK_ARG(T >= 1 && k >= 1 && k <= 256 && rows >= 1 && H >= 1);
  MOE_CHECK_ARG(n_tokens >= 1 && (token_ids != nullptr || n_tokens >= T));
  MOE_CHECK_ARG(accumulate == 0 || accumulate == 1);
  MOE_CHECK_ARG(slot_of_expert == nullptr || (E >= 1 && E <= 256));
  if (dtype == MOE_BF16 && H % 8 != 0) return MOE_ERR_UNSUPPORTED;
  if (dtype == MOE_F32 && H % 4 != 0) return MOE_ERR_UNSUPPORTED;
  const int64_t blocks = ceil_div(T, kCombWaves);
  if (blocks > 0x7fffffff) return MOE_ERR_UNSUPPORTED;
  CombArgs a{y_perm, H, rows, token_ids, T, n_tokens, k, topk_idx, topk_w, row_of_pair,
             slot_of_expert, E, y_shared, accumulate, y, incomplete};
  hipStream_t st = as_stream(stream);
  if (dtype == MOE_BF16 && k <= 8) {
    const dim3 g((unsigned)blocks), b(kCombWaves * kWave);
    if (k <= 2) combine_bf16_kernel<2><<<g, b, 0, st>>>(a);
    else if (k <= 4) combine_bf16_kernel<4><<<g, b, 0, st>>>(a);
    else combine_bf16_kernel<8><<<g, b, 0, st>>>(a);
  } else if (dtype == MOE_BF16)
    combine_kernel<true><<<dim3((unsigned)blocks), dim3(kCombWaves * kWave), 0, st>>>(a);
  else
    combine_kernel<false><<<dim3((unsigned)blocks), dim3(kCombWaves * kWave), 0, st>>>(a);
  MOE_CHECK_LAUNCH();
  return MOE_OK;
}
