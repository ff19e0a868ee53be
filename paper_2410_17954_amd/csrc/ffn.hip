// moe_expert_ffn: grouped SwiGLU experts (Sec. 2.1) over the experts that the
// slot table marks as resident in the expert cache (Sec. 3.4).
//
// bf16 path: two grouped GEMMs on MFMA (v_mfma_f32_32x32x16_bf16), both of the
// form C[rows of expert e, :] = A[rows, K] . B_s[N, K]^T with K contiguous in
// both operands:
//   up   : A = x_perm, B = the gate and up projections of slot s, interleaved
//          in 32-row groups so that one wave holds gate and up accumulators
//          for the same (row, f); the epilogue writes a = silu(g) * u as bf16;
//   down : A = a, B = the down projection of slot s; the epilogue writes bf16.
// The grid is persistent (one block per compute unit); tile t is mapped so
// that each XCD (blocks b with the same b % 8) works on a contiguous range of
// tiles: the row tiles of one expert that share a weight tile then run
// together and share it through that XCD's L2. A small prologue kernel turns
// expert_offsets and the slot table into a prefix of row tiles per resident
// expert; everything stays on the device.
// Fast path (H and F multiples of 32): `ffn_gemm_bf16_v2`, 256 x 256 x 32
// tiles, 8 waves, a four-stage LDS ring filled by direct global->LDS DMA.
// General path (H, F multiples of 8): `ffn_gemm_bf16`, 256 x 128 x 64 tiles,
// 4 waves, register-staged LDS double buffer with zero-filled K tails.
//
// f32 path (small, correctness-oriented): one thread per output element.
#include "common.h"

#include <math.h>

#include <type_traits>

namespace moe {
namespace {

constexpr int BM = 256;
constexpr int BN = 128;
constexpr int BK = 64;
constexpr int kThreads = 256;
constexpr int kChunks = BK / 8;           // 16-byte K-chunks per tile row

// Per-expert row-tile prefix of resident experts; also clears the per-XCD
// tile-claim counters of the two GEMMs (kClaimWords ints after prefix[E]).
constexpr int kClaimWords = 16;
__global__ void ffn_tiles_kernel(const int32_t* __restrict__ offsets,
                                 const int32_t* __restrict__ slot, int E, int S,
                                 int64_t max_rows, int bm, int32_t* __restrict__ prefix) {
  if (blockIdx.x != 0) return;
  if (threadIdx.x < kClaimWords) prefix[E + 1 + threadIdx.x] = 0;
  if (threadIdx.x != 0) return;
  int32_t run = 0;
  for (int e = 0; e < E; ++e) {
    prefix[e] = run;
    const int s = slot ? slot[e] : e;
    int64_t lo = offsets[e], hi = offsets[e + 1];
    lo = lo < 0 ? 0 : (lo > max_rows ? max_rows : lo);
    hi = hi < lo ? lo : (hi > max_rows ? max_rows : hi);
    if (s >= 0 && s < S) run += (int32_t)((hi - lo + bm - 1) / bm);
  }
  prefix[E] = run;
}

__device__ __forceinline__ int swz(int row, int chunk) {
  return chunk ^ ((row >> 1) & 7);
}

// EPI 0: SwiGLU up projection, EPI 1: down projection.
template <int EPI>
__global__ void __launch_bounds__(kThreads, 1)
ffn_gemm_bf16(const uint16_t* __restrict__ A, int64_t K,
              const uint16_t* __restrict__ B0, const uint16_t* __restrict__ B1,
              int64_t F, int64_t H,
              const int32_t* __restrict__ offsets, const int32_t* __restrict__ slot,
              int E, int64_t max_rows, const int32_t* __restrict__ prefix,
              uint16_t* __restrict__ C) {
  // EPI 0: N of the output = F (a block covers 64 f, as 64 gate + 64 up rows)
  // EPI 1: N of the output = H (a block covers 128 h)
  constexpr int kOutN = EPI == 0 ? BN / 2 : BN;
  const int64_t N_out = EPI == 0 ? F : H;
  const int64_t ldc = N_out;
  const int64_t n_tiles = (N_out + kOutN - 1) / kOutN;

  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * BK];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * BK];

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid / kWave;
  const int wm = wave >> 1, wn = wave & 1;

  const int64_t total = (int64_t)prefix[E] * n_tiles;
  const int64_t G = gridDim.x;               // multiple of 8
  const int64_t per_xcd = G / 8;
  const int64_t first = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;

  for (int64_t t = first; t < total; t += G) {
    // ---- decode tile -> (expert, row tile, column tile)
    int e = 0;
    while (e + 1 < E && (int64_t)prefix[e + 1] * n_tiles <= t) ++e;
    const int64_t local = t - (int64_t)prefix[e] * n_tiles;
    const int64_t me = prefix[e + 1] - prefix[e];
    const int64_t nt = local / me;
    const int64_t mt = local - nt * me;
    const int s = slot ? slot[e] : e;
    int64_t lo = offsets[e];
    lo = lo < 0 ? 0 : (lo > max_rows ? max_rows : lo);
    int64_t hi = offsets[e + 1];
    hi = hi < lo ? lo : (hi > max_rows ? max_rows : hi);
    const int64_t row0 = lo + mt * BM;
    const int64_t row_end = min(row0 + (int64_t)BM, hi);
    const int64_t n0 = nt * kOutN;

    // ---- per-thread global source pointers for the staged loads
    // A: 256 rows x 8 chunks = 2048 chunks, 8 per thread (rows tid/8 + 32 i)
    // B: 128 rows x 8 chunks = 1024 chunks, 4 per thread
    const int lrow = tid / kChunks;
    const int lch = tid % kChunks;
    const uint16_t* a_src[8];
    bool a_ok[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int64_t r = row0 + lrow + 32 * i;
      a_ok[i] = r < row_end;
      a_src[i] = A + (a_ok[i] ? r : row0) * K + lch * 8;
    }
    const uint16_t* b_src[4];
    bool b_ok[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int n = lrow + 32 * i;          // virtual B row in the tile
      int64_t wrow;
      const uint16_t* base;
      if (EPI == 0) {
        const int grp = n >> 5;             // 32-row groups: gate, up, gate, up
        const int64_t f = n0 + (grp >> 1) * 32 + (n & 31);
        b_ok[i] = f < F;
        base = ((grp & 1) ? B1 : B0) + (int64_t)s * F * H;
        wrow = b_ok[i] ? f : 0;
      } else {
        const int64_t h = n0 + n;
        b_ok[i] = h < H;
        base = B0 + (int64_t)s * H * F;
        wrow = b_ok[i] ? h : 0;
      }
      b_src[i] = base + wrow * K + lch * 8;
    }

    f32x16_t acc[4][2];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[mi][ni][q] = 0.f;

    uint4 ra[8], rb[4];
    auto gload = [&](int64_t k0) {
      const bool kin = k0 + lch * 8 < K;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        ra[i] = (a_ok[i] && kin) ? *reinterpret_cast<const uint4*>(a_src[i] + k0)
                                 : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int i = 0; i < 4; ++i)
        rb[i] = (b_ok[i] && kin) ? *reinterpret_cast<const uint4*>(b_src[i] + k0)
                                 : make_uint4(0, 0, 0, 0);
    };
    auto sstore = [&](int buf) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int r = lrow + 32 * i;
        *reinterpret_cast<uint4*>(&As[buf][r * BK + swz(r, lch) * 8]) = ra[i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = lrow + 32 * i;
        *reinterpret_cast<uint4*>(&Bs[buf][r * BK + swz(r, lch) * 8]) = rb[i];
      }
    };

    const int64_t ktiles = (K + BK - 1) / BK;
    gload(0);
    sstore(0);
    __syncthreads();

    const int frow = lane & 31;         // fragment row within a 32-row MFMA tile
    const int fk = lane >> 5;           // which 8-wide half of the 16-wide K step
    for (int64_t kt = 0; kt < ktiles; ++kt) {
      const int buf = kt & 1;
      if (kt + 1 < ktiles) gload((kt + 1) * BK);
      const uint16_t* as = As[buf];
      const uint16_t* bs = Bs[buf];
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        const int ch = ks * 2 + fk;
        bf16x8_t af[4], bfr[2];
#pragma unroll
        for (int mi = 0; mi < 4; ++mi) {
          const int r = wm * 128 + mi * 32 + frow;
          af[mi] = *reinterpret_cast<const bf16x8_t*>(&as[r * BK + swz(r, ch) * 8]);
        }
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) {
          const int r = wn * 64 + ni * 32 + frow;
          bfr[ni] = *reinterpret_cast<const bf16x8_t*>(&bs[r * BK + swz(r, ch) * 8]);
        }
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
          for (int ni = 0; ni < 2; ++ni)
            acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mi], bfr[ni], acc[mi][ni], 0, 0, 0);
      }
      if (kt + 1 < ktiles) sstore(buf ^ 1);
      __syncthreads();
    }

    // ---- epilogue. 32x32 C layout: lane holds column lane % 32 and rows
    // 8 * (q / 4) + 4 * (lane / 32) + (q % 4) for q = 0..15.
    const int ccol = lane & 31;
    const int crow = (lane >> 5) * 4;
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) {
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int64_t r = row0 + wm * 128 + mi * 32 + 8 * (q >> 2) + crow + (q & 3);
        if (r >= row_end) continue;
        if (EPI == 0) {
          const int64_t f = n0 + wn * 32 + ccol;
          if (f < F) {
            const float g = acc[mi][0][q];
            const float u = acc[mi][1][q];
            const float act = g / (1.f + expf(-g)) * u;
            C[r * ldc + f] = f32_to_bf16(act);
          }
        } else {
#pragma unroll
          for (int ni = 0; ni < 2; ++ni) {
            const int64_t h = n0 + wn * 64 + ni * 32 + ccol;
            if (h < H) C[r * ldc + h] = f32_to_bf16(acc[mi][ni][q]);
          }
        }
      }
    }
  }
}

// ------------------------------------------------------- bf16 fast path
// 256 x 256 tiles, 8 waves (2 per SIMD) in a 2 (M) x 4 (N) arrangement, each
// wave 128 x 64 of the output (4 x 2 MFMA 32x32x16 tiles). Operands move from
// global memory straight into LDS (global_load_lds_dwordx4: each lane deposits
// 16 bytes at M0 + 16 * lane), so no registers are spent on staging; the XOR
// swizzle is applied on the load side by choosing which K-chunk each lane
// fetches. A ring of STAGES LDS stages of BK-deep tiles keeps STAGES-1 steps
// of loads in flight while one step is multiplied; at the end of a step each
// wave waits only for the loads of the next step, then one barrier.
// Needs K % BK == 0.
namespace v2 {
constexpr int BM = 256, BN = 256;
constexpr int kWaves = 8, kThreads = kWaves * 64;
constexpr int FAST_BK = 32, FAST_STAGES = 4;
}  // namespace v2

typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ void lds_dma16(const void* g, void* lds_wave_base) {
  __builtin_amdgcn_global_load_lds(g, (lds_void*)lds_wave_base, 16, 0, 0);
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt_hi[15:14]).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

template <int EPI, int BK, int STAGES>
__global__ void __launch_bounds__(v2::kThreads, 1)
ffn_gemm_bf16_v2(const uint16_t* __restrict__ A, int64_t K,
                 const uint16_t* __restrict__ B0, const uint16_t* __restrict__ B1,
                 int64_t F, int64_t H,
                 const int32_t* __restrict__ offsets, const int32_t* __restrict__ slot,
                 int E, int64_t max_rows, const int32_t* __restrict__ prefix,
                 int32_t* __restrict__ claim, uint16_t* __restrict__ C) {
  constexpr int BM = v2::BM, BN = v2::BN;
  constexpr int CPR = BK / 8;                  // 16-byte chunks per tile row
  constexpr int RPW = 128 / BK;                // rows per 256-byte bank window
  constexpr int ROWS_PER_PIECE = 512 / BK;     // rows per 1 KB DMA piece
  constexpr int PIECES = BM * BK / 512;        // 1 KB pieces per operand stage
  constexpr int PPW = PIECES / v2::kWaves;     // pieces per wave per operand
  constexpr int kStageA = BM * BK, kStageB = BN * BK;   // elements
  constexpr int kOutN = EPI == 0 ? BN / 2 : BN;
  static_assert(PPW * v2::kWaves == PIECES, "piece split");
  static_assert((STAGES * (kStageA + kStageB) * 2) <= 160 * 1024, "LDS");

  const int64_t N_out = EPI == 0 ? F : H;
  const int64_t ldc = N_out;
  const int64_t n_tiles = (N_out + kOutN - 1) / kOutN;

  // One LDS object per stage: the compiler then proves that a DMA into one
  // stage cannot alias reads of another and inserts no blanket vmcnt(0).
  static_assert(STAGES == 4, "four LDS stages");
  __shared__ __attribute__((aligned(1024))) uint16_t As0[kStageA], As1[kStageA], As2[kStageA], As3[kStageA];
  __shared__ __attribute__((aligned(1024))) uint16_t Bs0[kStageB], Bs1[kStageB], Bs2[kStageB], Bs3[kStageB];
  uint16_t* const As[4] = {As0, As1, As2, As3};
  uint16_t* const Bs[4] = {Bs0, Bs1, Bs2, Bs3};

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid / kWave;
  const int wm = wave >> 2, wn = wave & 3;    // 2 x 4 waves

  const int64_t total = (int64_t)prefix[E] * n_tiles;
  const int64_t per_xcd = gridDim.x / 8;        // blocks per XCD = tiles per chunk
  const int xcd = blockIdx.x % 8;
  const int64_t ktiles = K / BK;
  __shared__ int64_t s_claim;

  const int lrow = lane / CPR;                // row within a DMA piece
  const int lpch = lane % CPR;                // physical chunk this lane fills
  auto swz = [](int r, int c) { return c ^ ((r / RPW) % CPR); };

  // Tiles are claimed dynamically from a per-XCD counter: the j-th claim on
  // XCD x takes tile ((j / C) * 8 + x) * C + j % C (C = blocks per XCD), so
  // each XCD walks its own chunks of C consecutive tiles, and blocks that
  // drew cheap (partly empty) tiles simply claim more.
  for (;;) {
    if (tid == 0) s_claim = atomicAdd(&claim[xcd], 1);
    __syncthreads();
    const int64_t j = s_claim;
    const int64_t t = ((j / per_xcd) * 8 + xcd) * per_xcd + (j % per_xcd);
    if (t >= total) break;
    int e = 0;
    while (e + 1 < E && (int64_t)prefix[e + 1] * n_tiles <= t) ++e;
    const int64_t local = t - (int64_t)prefix[e] * n_tiles;
    const int64_t me = prefix[e + 1] - prefix[e];
    const int64_t nt = local / me;
    const int64_t mt = local - nt * me;
    const int s = slot ? slot[e] : e;
    int64_t lo = offsets[e];
    lo = lo < 0 ? 0 : (lo > max_rows ? max_rows : lo);
    int64_t hi = offsets[e + 1];
    hi = hi < lo ? lo : (hi > max_rows ? max_rows : hi);
    const int64_t row0 = lo + mt * BM;
    const int64_t row_end = min(row0 + (int64_t)BM, hi);
    const int64_t n0 = nt * kOutN;
    // A wave whose 128-row half holds no row of the expert skips its LDS reads
    // and MFMAs (it still takes part in loads and barriers), so a tile with at
    // most 128 rows costs about half.
    const bool active = __builtin_amdgcn_readfirstlane((int)(row_end - row0 > wm * 128)) != 0;

    // Per-lane source pointers (the K offset is added per step). Rows past the
    // end of the expert (or of the weight) read a valid row; their results are
    // never stored.
    const uint16_t* a_src[PPW];
    const uint16_t* b_src[PPW];
#pragma unroll
    for (int i = 0; i < PPW; ++i) {
      const int r = (wave * PPW + i) * ROWS_PER_PIECE + lrow;   // tile row
      const int lch = swz(r, lpch);                              // logical chunk
      int64_t ar = row0 + r;
      if (ar >= row_end) ar = row0;
      a_src[i] = A + ar * K + lch * 8;
      int64_t wrow;
      const uint16_t* base;
      if (EPI == 0) {
        const int grp = r >> 5;                  // 32-row groups: gate, up, gate, up, ...
        int64_t f = n0 + (grp >> 1) * 32 + (r & 31);
        if (f >= F) f = 0;
        base = ((grp & 1) ? B1 : B0) + (int64_t)s * F * H;
        wrow = f;
      } else {
        int64_t h = n0 + r;
        if (h >= H) h = 0;
        base = B0 + (int64_t)s * H * F;
        wrow = h;
      }
      b_src[i] = base + wrow * K + lch * 8;
    }
    auto issue = [&](auto stage_c, int64_t step) {
      constexpr int stage = decltype(stage_c)::value;
      const int64_t k0 = step * BK;
#pragma unroll
      for (int i = 0; i < PPW; ++i) {
        lds_dma16(a_src[i] + k0, As[stage] + (wave * PPW + i) * 512);
        lds_dma16(b_src[i] + k0, Bs[stage] + (wave * PPW + i) * 512);
      }
    };

    f32x16_t acc[4][2];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[mi][ni][q] = 0.f;

    // prologue: STAGES-1 steps in flight, the first one complete
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using I3 = std::integral_constant<int, 3>;
    if (0 < ktiles) issue(I0{}, 0);
    if (1 < ktiles) issue(I1{}, 1);
    if (2 < ktiles) issue(I2{}, 2);
    {
      const int64_t inflight = min((int64_t)STAGES - 1, ktiles) - 1;   // beyond step 0
      if (inflight >= 2) wait_vmcnt<2 * 2 * PPW>();
      else if (inflight == 1) wait_vmcnt<2 * PPW>();
      else wait_vmcnt<0>();
    }
    __syncthreads();

    const int frow = lane & 31;
    const int fk = lane >> 5;
    // One K-step on stage J: start the loads of step kt+3 into stage J+3
    // (mod 4), multiply stage J, wait for step kt+1, barrier.
    auto step = [&](auto j_c, int64_t kt) {
      constexpr int J = decltype(j_c)::value;
      if (kt + STAGES - 1 < ktiles)
        issue(std::integral_constant<int, (J + STAGES - 1) % STAGES>{}, kt + STAGES - 1);
      const uint16_t* as = As[J];
      const uint16_t* bs = Bs[J];
      // All fragments of the step first (BK/16 substeps x 6 reads), then the
      // MFMAs, so LDS latency overlaps the matrix work.
      constexpr int KS = BK / 16;
      bf16x8_t af[KS][4], bfr[KS][2];
      if (active) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const int ch = ks * 2 + fk;
#pragma unroll
          for (int mi = 0; mi < 4; ++mi) {
            const int r = wm * 128 + mi * 32 + frow;
            af[ks][mi] = *reinterpret_cast<const bf16x8_t*>(&as[r * BK + swz(r, ch) * 8]);
          }
#pragma unroll
          for (int ni = 0; ni < 2; ++ni) {
            const int r = wn * 64 + ni * 32 + frow;
            bfr[ks][ni] = *reinterpret_cast<const bf16x8_t*>(&bs[r * BK + swz(r, ch) * 8]);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int mi = 0; mi < 4; ++mi)
#pragma unroll
            for (int ni = 0; ni < 2; ++ni)
              acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[ks][mi], bfr[ks][ni], acc[mi][ni], 0, 0, 0);
      }
      // Wait for the loads of step kt+1 only; later steps stay in flight.
      const int64_t later = min(kt + STAGES - 1, ktiles - 1) - (kt + 1);
      if (later >= 2) wait_vmcnt<2 * 2 * PPW>();
      else if (later == 1) wait_vmcnt<2 * PPW>();
      else wait_vmcnt<0>();
      __syncthreads();
    };
    int64_t kt = 0;
    for (; kt + STAGES <= ktiles; kt += STAGES) {
      step(I0{}, kt);
      step(I1{}, kt + 1);
      step(I2{}, kt + 2);
      step(I3{}, kt + 3);
    }
    if (kt < ktiles) step(I0{}, kt);
    if (kt + 1 < ktiles) step(I1{}, kt + 1);
    if (kt + 2 < ktiles) step(I2{}, kt + 2);

    // Epilogue (32x32 C layout: column lane % 32, rows 8*(q/4) + 4*(lane/32) + q%4).
    const int ccol = lane & 31;
    const int crow = (lane >> 5) * 4;
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) {
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int64_t r = row0 + wm * 128 + mi * 32 + 8 * (q >> 2) + crow + (q & 3);
        if (r >= row_end) continue;
        if (EPI == 0) {
          const int64_t f = n0 + wn * 32 + ccol;
          if (f < F) {
            const float g = acc[mi][0][q];
            const float u = acc[mi][1][q];
            C[r * ldc + f] = f32_to_bf16(g / (1.f + expf(-g)) * u);
          }
        } else {
#pragma unroll
          for (int ni = 0; ni < 2; ++ni) {
            const int64_t h = n0 + wn * 64 + ni * 32 + ccol;
            if (h < H) C[r * ldc + h] = f32_to_bf16(acc[mi][ni][q]);
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------- f32 path
__device__ __forceinline__ int expert_of_row(const int32_t* offsets, int E, int64_t r) {
  // last e with offsets[e] <= r (offsets non-decreasing)
  int lo = 0, hi = E;  // answer in [0, E)
  while (hi - lo > 1) {
    const int mid = (lo + hi) / 2;
    if (offsets[mid] <= r) lo = mid; else hi = mid;
  }
  return lo;
}

__global__ void ffn_f32_up(const float* __restrict__ x, int64_t H, int64_t F,
                           const int32_t* __restrict__ offsets, const int32_t* __restrict__ slot,
                           int E, int S, int64_t max_rows, const float* __restrict__ wg,
                           const float* __restrict__ wu, float* __restrict__ act) {
  const int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int64_t r = q / F, f = q % F;
  if (r >= max_rows) return;
  const int64_t end = min((int64_t)offsets[E], max_rows);
  if (r < offsets[0] || r >= end) return;
  const int e = expert_of_row(offsets, E, r);
  const int s = slot ? slot[e] : e;
  if (s < 0 || s >= S) return;
  const float* xr = x + r * H;
  const float* g = wg + ((int64_t)s * F + f) * H;
  const float* u = wu + ((int64_t)s * F + f) * H;
  float sg = 0.f, su = 0.f;
  for (int64_t h = 0; h < H; ++h) {
    sg = fmaf(xr[h], g[h], sg);
    su = fmaf(xr[h], u[h], su);
  }
  act[r * F + f] = sg / (1.f + expf(-sg)) * su;
}

__global__ void ffn_f32_down(const float* __restrict__ act, int64_t H, int64_t F,
                             const int32_t* __restrict__ offsets, const int32_t* __restrict__ slot,
                             int E, int S, int64_t max_rows, const float* __restrict__ wd,
                             float* __restrict__ y) {
  const int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int64_t r = q / H, h = q % H;
  if (r >= max_rows) return;
  const int64_t end = min((int64_t)offsets[E], max_rows);
  if (r < offsets[0] || r >= end) return;
  const int e = expert_of_row(offsets, E, r);
  const int s = slot ? slot[e] : e;
  if (s < 0 || s >= S) return;
  const float* ar = act + r * F;
  const float* d = wd + ((int64_t)s * H + h) * F;
  float acc = 0.f;
  for (int64_t f = 0; f < F; ++f) acc = fmaf(ar[f], d[f], acc);
  y[r * H + h] = acc;
}

}  // namespace
}  // namespace moe

extern "C" size_t moe_expert_ffn_workspace(int64_t max_rows, int64_t H, int64_t F, int32_t E,
                                           int32_t dtype) {
  (void)H;
  if (max_rows < 1 || F < 1 || E < 1 || !moe::valid_dtype(dtype)) return 0;
  const size_t elt = dtype == MOE_BF16 ? 2 : 4;
  size_t bytes = moe::align_up((size_t)max_rows * (size_t)F * elt, 256);
  bytes += moe::align_up((size_t)(E + 1 + 16) * sizeof(int32_t), 256);
  return bytes;
}

extern "C" int moe_expert_ffn(const void* x_perm, int32_t dtype, int64_t max_rows, int64_t H,
                              int64_t F, const int32_t* expert_offsets, int32_t E,
                              const int32_t* slot_of_expert, int32_t S, const void* w_gate,
                              const void* w_up, const void* w_down, void* y_perm,
                              void* workspace, size_t ws_bytes, void* stream) {
  using namespace moe;
  MOE_CHECK_ARG(x_perm && expert_offsets && y_perm);
  MOE_CHECK_ARG(valid_dtype(dtype));
  MOE_CHECK_ARG(max_rows >= 1 && H >= 1 && F >= 1 && E >= 1 && E <= 256 && S >= 0);
  MOE_CHECK_ARG(slot_of_expert != nullptr || S >= E);
  MOE_CHECK_ARG(S == 0 || (w_gate && w_up && w_down));
  MOE_CHECK_ARG(max_rows < ((int64_t)1 << 31));
  if (dtype == MOE_BF16 && (H % 8 != 0 || F % 8 != 0)) return MOE_ERR_UNSUPPORTED;
  const size_t need = moe_expert_ffn_workspace(max_rows, H, F, E, dtype);
  if (!workspace || ws_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255))
    return MOE_ERR_WORKSPACE;
  if (S == 0) return MOE_OK;  // nothing resident: every row is a miss
  hipStream_t st = as_stream(stream);
  const size_t elt = dtype == MOE_BF16 ? 2 : 4;
  char* ws = static_cast<char*>(workspace);
  void* act = ws;
  int32_t* prefix = reinterpret_cast<int32_t*>(ws + align_up((size_t)max_rows * F * elt, 256));

  if (dtype == MOE_F32) {
    const int64_t n1 = max_rows * F, n2 = max_rows * H;
    if (ceil_div(n1, 256) > 0x7fffffff || ceil_div(n2, 256) > 0x7fffffff) return MOE_ERR_UNSUPPORTED;
    ffn_f32_up<<<dim3((unsigned)ceil_div(n1, 256)), dim3(256), 0, st>>>(
        static_cast<const float*>(x_perm), H, F, expert_offsets, slot_of_expert, E, S, max_rows,
        static_cast<const float*>(w_gate), static_cast<const float*>(w_up), static_cast<float*>(act));
    MOE_CHECK_LAUNCH();
    ffn_f32_down<<<dim3((unsigned)ceil_div(n2, 256)), dim3(256), 0, st>>>(
        static_cast<const float*>(act), H, F, expert_offsets, slot_of_expert, E, S, max_rows,
        static_cast<const float*>(w_down), static_cast<float*>(y_perm));
    MOE_CHECK_LAUNCH();
    return MOE_OK;
  }

  const bool fast = (H % v2::FAST_BK == 0) && (F % v2::FAST_BK == 0);
  const int bm = fast ? v2::BM : BM;
  ffn_tiles_kernel<<<dim3(1), dim3(64), 0, st>>>(expert_offsets, slot_of_expert, E, S, max_rows,
                                                 bm, prefix);
  MOE_CHECK_LAUNCH();
  int grid = device_cu_count();
  grid = (grid + 7) / 8 * 8;
  const auto* xb = static_cast<const uint16_t*>(x_perm);
  auto* ab = static_cast<uint16_t*>(act);
  const auto* wgb = static_cast<const uint16_t*>(w_gate);
  const auto* wub = static_cast<const uint16_t*>(w_up);
  const auto* wdb = static_cast<const uint16_t*>(w_down);
  auto* yb = static_cast<uint16_t*>(y_perm);
  if (fast) {
    ffn_gemm_bf16_v2<0, v2::FAST_BK, v2::FAST_STAGES><<<dim3(grid), dim3(v2::kThreads), 0, st>>>(
        xb, H, wgb, wub, F, H, expert_offsets, slot_of_expert, E, max_rows, prefix,
        prefix + E + 1, ab);
    MOE_CHECK_LAUNCH();
    ffn_gemm_bf16_v2<1, v2::FAST_BK, v2::FAST_STAGES><<<dim3(grid), dim3(v2::kThreads), 0, st>>>(
        ab, F, wdb, nullptr, F, H, expert_offsets, slot_of_expert, E, max_rows, prefix,
        prefix + E + 1 + 8, yb);
    MOE_CHECK_LAUNCH();
    return MOE_OK;
  }
  ffn_gemm_bf16<0><<<dim3(grid), dim3(kThreads), 0, st>>>(
      xb, H, wgb, wub, F, H, expert_offsets, slot_of_expert, E, max_rows, prefix, ab);
  MOE_CHECK_LAUNCH();
  ffn_gemm_bf16<1><<<dim3(grid), dim3(kThreads), 0, st>>>(
      ab, F, wdb, nullptr, F, H, expert_offsets, slot_of_expert, E, max_rows, prefix, yb);
  MOE_CHECK_LAUNCH();
  return MOE_OK;
}
