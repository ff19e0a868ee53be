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
// Fast path (H and F multiples of 32): `ffn_gemm_bf16_fast`, 256 x 256 x 32
// tiles, 4 waves of 128 x 128, a four-stage LDS ring filled by direct
// global->LDS DMA.
// General path (H, F multiples of 8): `ffn_gemm_bf16`, 256 x 128 x 64 tiles,
// 4 waves, register-staged LDS double buffer with zero-filled K tails.
//
// f32 path (small, correctness-oriented): one thread per output element.
#include "common.h"

#include <math.h>

#include <algorithm>
#include <type_traits>

namespace moe {
namespace {

constexpr int BM = 256;
constexpr int BN = 128;
constexpr int BK = 64;
constexpr int kThreads = 256;
constexpr int kChunks = BK / 8;           // 16-byte K-chunks per tile row

// Counters after prefix[E]: 16 per-XCD tile claims (8 per GEMM), then per
// GEMM one claim counter for the split tail and kMaxTailTiles arrival
// counters (one per tail tile).
constexpr int kClaimWords = 16;
constexpr int kMaxTailTiles = 1024;
constexpr int kTailWords = 1 + kMaxTailTiles;
constexpr int kCounterWords = kClaimWords + 2 * kTailWords;

// Per-expert row-tile prefix of resident experts; also clears the counters.
// Resident experts with at most 16 * small_tiles rows (small_tiles 0 or
// kSmallMaxTiles) get no row tiles here: they are listed for the few-row
// kernel instead (small[0] = their number, small[1..] = their ids, those with
// the most 16-row tiles first, ascending ids within a tile count).
// With split_small an expert's last row tile, when it holds at most bm / 8
// rows, is counted apart (prefix2: 0 or 1 per expert), so that the GEMMs can
// run every expert's full-cost row tiles first and these small ones last: a
// tile that short runs its K loop several times faster than the full tiles
// beside it, so kept in its column group it runs ahead of the tiles that share
// its weights in L2 and streams them from HBM alone. A last tile of more than
// bm / 8 rows keeps close enough pace to stay in place.
constexpr int kSmallMaxTiles = 6;              // few-row experts: at most 96 rows

__global__ void ffn_tiles_kernel(const int32_t* __restrict__ offsets,
                                 const int32_t* __restrict__ slot, int E, int S,
                                 int64_t max_rows, int bm, int small_tiles, int split_small,
                                 int32_t* __restrict__ prefix) {
  if (blockIdx.x != 0) return;
  for (int q = threadIdx.x; q < kCounterWords; q += blockDim.x) prefix[E + 1 + q] = 0;
  if (threadIdx.x != 0) return;
  int32_t* const small = prefix + E + 1 + kCounterWords;
  int32_t* const prefix2 = small + E + 1;
  int32_t run = 0, run2 = 0;
  int32_t n_of[kSmallMaxTiles + 1] = {};
  auto rows_of = [&](int e) -> int64_t {
    const int s = slot ? slot[e] : e;
    int64_t lo = offsets[e], hi = offsets[e + 1];
    lo = lo < 0 ? 0 : (lo > max_rows ? max_rows : lo);
    hi = hi < lo ? lo : (hi > max_rows ? max_rows : hi);
    return (s < 0 || s >= S) ? 0 : hi - lo;
  };
  for (int e = 0; e < E; ++e) {
    prefix[e] = run;
    prefix2[e] = run2;
    const int64_t m = rows_of(e);
    if (m == 0) continue;
    if (m <= 16 * small_tiles) {
      ++n_of[(m + 15) / 16];
    } else {
      const int64_t nt = (m + bm - 1) / bm;
      if (split_small && m - (nt - 1) * bm <= bm / 8) {
        run += (int32_t)(nt - 1);
        ++run2;
      } else {
        run += (int32_t)nt;
      }
    }
  }
  prefix[E] = run;
  prefix2[E] = run2;
  // few-row experts by descending tile count: the grid strides over their
  // units in list order, so the costliest units start first
  int32_t at[kSmallMaxTiles + 1];
  int32_t n = 0;
  for (int c = kSmallMaxTiles; c >= 1; --c) {
    at[c] = n;
    n += n_of[c];
  }
  small[0] = n;
  if (n == 0) return;
  for (int e = 0; e < E; ++e) {
    const int64_t m = rows_of(e);
    if (m > 0 && m <= 16 * small_tiles) small[1 + at[(m + 15) / 16]++] = e;
  }
}

// silu(g) * u with the hardware exp2 and reciprocal (about 2 ulp of float32,
// far below the bf16 rounding of the result); exp2 overflows to +inf for very
// negative g, giving g * 0 * u = -0 as the exact expression does.
__device__ __forceinline__ float swiglu(float g, float u) {
  const float e = __builtin_amdgcn_exp2f(-g * 1.4426950408889634f);
  return g * __builtin_amdgcn_rcpf(1.f + e) * u;
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
            const float act = swiglu(g, u);
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

// ------------------------------------------------------- few rows per expert
// An expert with at most 16 * kSmallMaxTiles rows (decode-sized batches) is
// bound by reading its weights once, not by MFMA. A block of four waves owns
// one unit: SmallShape<EPI>::COLS output columns (weight rows) of one such
// expert, all of its rows; wave w streams the w-th quarter of the K range of
// those weight rows with 16x16x32 MFMAs (the expert's rows padded to 16 * MT,
// MT = ceil(rows / 16)), and the four partial sums are added through LDS.
// Splitting K inside the block, rather than giving each wave its own columns,
// keeps the addresses the whole chip reads at one time close together, which
// DRAM serves faster. A unit has four 16-column tiles of weights per K step
// (gate and up of 32 columns, or 64 columns of the down projection), so the
// activation fragments a wave loads (again in every unit of the expert, from
// L2) are MT/4 of its weight loads; those extra load instructions, not the
// MFMAs, are what slows the unit as MT grows.
constexpr int kSmallWaves = 4;
constexpr int kSmallRC = 2;                      // row tiles per LDS reduction pass

template <int EPI>
struct SmallShape {
  static constexpr int NB = EPI == 0 ? 2 : 1;    // gate and up, or down
  static constexpr int NT = 4 / NB;              // 16-column MFMA tiles per unit
  static constexpr int COLS = 16 * NT;
};
// K steps of 32 loaded per batch: four while the rows' fragments are few,
// two for three or more row tiles (registers)
template <int MT>
constexpr int small_unroll() { return MT <= 2 ? 4 : 2; }

// MTMAX: the most row tiles of any listed expert the launch supports; each
// unit takes the body for its expert's tile count (uniform per block).
template <int EPI, int MTMAX>
__global__ void __launch_bounds__(64 * kSmallWaves) __attribute__((amdgpu_waves_per_eu(2)))
ffn_small_bf16(const uint16_t* __restrict__ A, int64_t K, const uint16_t* __restrict__ B0,
               const uint16_t* __restrict__ B1, int64_t F, int64_t H,
               const int32_t* __restrict__ offsets, const int32_t* __restrict__ slot,
               int64_t max_rows, const int32_t* __restrict__ small, uint16_t* __restrict__ C) {
  using SS = SmallShape<EPI>;
  constexpr int NB = SS::NB, NT = SS::NT;
  constexpr int RC = MTMAX < kSmallRC ? MTMAX : kSmallRC;
  __shared__ f32x4_t part[kSmallWaves][RC][NT][NB][kWave];
  const int64_t N_out = EPI == 0 ? F : H;        // a multiple of 32 (fast path)
  const int ncb = (int)((N_out + SS::COLS - 1) / SS::COLS);
  const int64_t units = (int64_t)small[0] * ncb;
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int r = lane & 15;                       // A row / B column of this lane
  const int kq = (lane >> 4) * 8;                // its 8-wide slice of a K step
  const int64_t ks = K / 32;
  const int64_t per = (ks + kSmallWaves - 1) / kSmallWaves;
  const int64_t kb = min(ks, wave * per), ke = min(ks, kb + per);
  // byte offset of this lane's B slice from a weight tile's first row
  const uint32_t b_off = (uint32_t)(((int64_t)r * K + kq) * 2);
  auto run_unit = [&](auto mt_c, int e, int cb, int m, int64_t lo) {
    constexpr int MT = decltype(mt_c)::value;
    constexpr int U = small_unroll<MT>();
    const int s = slot ? slot[e] : e;
    const int64_t kfull = kb + (ke - kb) / U * U;
    const int64_t n0 = (int64_t)cb * SS::COLS;
    // wave-uniform bases plus 32-bit lane offsets. With one row tile, lanes of
    // rows past m load nothing (masked off, so no data comes back) and feed
    // zeros; with more, every lane loads (rows past m read the expert's last
    // row, whose products land in rows that are never stored): most of those
    // lanes are live, and the masks would cost registers.
    const char* const a_base = reinterpret_cast<const char*>(A + lo * K);
    uint32_t a_off[MT];
    bool a_on[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      a_on[i] = 16 * i + r < m;
      a_off[i] = (uint32_t)(((int64_t)min(16 * i + r, m - 1) * K + kq) * 2);
    }
    // a column tile past N_out (the last unit of a down projection whose
    // width is an odd multiple of 32) re-reads the unit's first tile and is
    // not stored
    const char* b_base[NT][NB];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const int64_t n = n0 + 16 * j < N_out ? n0 + 16 * j : n0;
      b_base[j][0] = reinterpret_cast<const char*>(B0 + ((int64_t)s * N_out + n) * K);
      if constexpr (EPI == 0)
        b_base[j][1] = reinterpret_cast<const char*>(B1 + ((int64_t)s * N_out + n) * K);
    }
    f32x4_t acc[MT][NT][NB];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int b = 0; b < NB; ++b) acc[i][j][b] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    auto steps = [&](int64_t s0, auto n_c) {
      constexpr int NS = decltype(n_c)::value;
      uint4 a[NS][MT], w[NS][NT][NB];
#pragma unroll
      for (int u = 0; u < NS; ++u) {
        const int64_t kbyte = (s0 + u) * 64;
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
          for (int b = 0; b < NB; ++b)
            w[u][j][b] = __builtin_bit_cast(uint4, __builtin_nontemporal_load(
                reinterpret_cast<const u32x4_t*>(b_base[j][b] + kbyte + b_off)));
#pragma unroll
        for (int i = 0; i < MT; ++i)
          a[u][i] = (MT > 1 || a_on[i]) ? *reinterpret_cast<const uint4*>(a_base + kbyte + a_off[i])
                                        : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < NS; ++u)
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
          for (int j = 0; j < NT; ++j)
#pragma unroll
            for (int b = 0; b < NB; ++b)
              acc[i][j][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                  __builtin_bit_cast(bf16x8_t, a[u][i]), __builtin_bit_cast(bf16x8_t, w[u][j][b]),
                  acc[i][j][b], 0, 0, 0);
    };
    for (int64_t s0 = kb; s0 < kfull; s0 += U) steps(s0, std::integral_constant<int, U>{});
    for (int64_t s0 = kfull; s0 < ke; ++s0) steps(s0, std::integral_constant<int, 1>{});
    // the four waves' partial sums, RC row tiles at a time: every wave writes
    // its own, then wave q adds up the (row tile, column tile) groups g with
    // g % 4 == q and stores them. C layout of the 16x16 MFMA: lane holds
    // column (lane % 16), rows 4 * (lane / 16) + q of its 16-row tile.
#pragma unroll
    for (int i0 = 0; i0 < MT; i0 += RC) {
#pragma unroll
      for (int ii = 0; ii < RC; ++ii)
        if (i0 + ii < MT)
#pragma unroll
          for (int j = 0; j < NT; ++j)
#pragma unroll
            for (int b = 0; b < NB; ++b) part[wave][ii][j][b][lane] = acc[i0 + ii][j][b];
      __syncthreads();
      const int groups = (MT - i0 < RC ? MT - i0 : RC) * NT;
      for (int g = wave; g < groups; g += kSmallWaves) {
        const int ii = g / NT, j = g % NT;
        const int64_t col = n0 + 16 * j + r;
        f32x4_t t[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          t[b] = part[0][ii][j][b][lane];
#pragma unroll
          for (int q = 1; q < kSmallWaves; ++q) t[b] += part[q][ii][j][b][lane];
        }
        if (col >= N_out) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int rr = 16 * (i0 + ii) + (lane >> 4) * 4 + q;
          if (rr >= m) continue;
          const float v = EPI == 0 ? swiglu(t[0][q], t[NB - 1][q]) : t[0][q];
          C[(lo + rr) * N_out + col] = f32_to_bf16(v);
        }
      }
      __syncthreads();                             // part is rewritten next
    }
  };
  // units (expert, column block) in list order, the grid striding over them:
  // at any time the blocks work on neighbouring columns
  for (int64_t unit = blockIdx.x; unit < units; unit += gridDim.x) {
    const int e = small[1 + (int)(unit / ncb)];
    const int cb = (int)(unit % ncb);
    int64_t lo = offsets[e], hi = offsets[e + 1];
    lo = lo < 0 ? 0 : (lo > max_rows ? max_rows : lo);
    hi = hi < lo ? lo : (hi > max_rows ? max_rows : hi);
    const int m = (int)(hi - lo);                  // 1 .. 16 * MTMAX (the list's rule)
    const int mt = (m + 15) / 16;
    if (mt <= 1) run_unit(std::integral_constant<int, 1>{}, e, cb, m, lo);
    else if (mt == 2) { if constexpr (MTMAX >= 2) run_unit(std::integral_constant<int, 2>{}, e, cb, m, lo); }
    else if (mt == 3) { if constexpr (MTMAX >= 3) run_unit(std::integral_constant<int, 3>{}, e, cb, m, lo); }
    else if (mt == 4) { if constexpr (MTMAX >= 4) run_unit(std::integral_constant<int, 4>{}, e, cb, m, lo); }
    else if (mt == 5) { if constexpr (MTMAX >= 5) run_unit(std::integral_constant<int, 5>{}, e, cb, m, lo); }
    else { if constexpr (MTMAX >= 6) run_unit(std::integral_constant<int, 6>{}, e, cb, m, lo); }
  }
}

// ------------------------------------------------------- LDS DMA helpers
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

// ------------------------------------------------------- bf16 fast path
// 256 x 256 block tiles, K in steps of 32, 4 waves (one per SIMD), each
// owning a 128 x 128 quarter of the output: 16 MFMA 32x32x16 accumulators,
// 256 registers, held in the accumulation registers. Per K-step a wave reads
// 128 + 128 rows of fragments from LDS for 2 x 128 x 128 x 32 flop, which
// keeps LDS traffic (fragment reads plus DMA writes) under the LDS bandwidth.
// Operands move from global memory straight into LDS
// (global_load_lds_dwordx4: each lane deposits 16 bytes at M0 + 16 * lane),
// with an XOR swizzle applied on the load side by choosing which K-chunk each
// lane fetches. A ring of four LDS stages keeps three K-steps of loads in
// flight. Within a step the second half-step's fragments are read while the
// first half's MFMAs run, then one barrier, then the next step's first
// fragments are read while the second half's MFMAs run. In each half the
// eight fragment reads go out within the first four MFMAs (so they have
// landed before the half ends) and the DMA of a later step (A pieces in the
// first half, B pieces in the second) is spread over the remaining twelve.
// A tile whose expert has at most 128 rows left is computed by all 4 waves
// side by side (each 32, 64 or 128 rows x 64 columns), so a ragged last row
// tile costs in proportion to its rows, on every SIMD.
// Needs K % 32 == 0.
namespace fast {
constexpr int BM = 256, BN = 256, BK = 32, STAGES = 4;
constexpr int kWaves = 4, kThreads = kWaves * 64;
constexpr int CPR = BK / 8;                 // 16-byte chunks per tile row
constexpr int RPW = 128 / BK;               // rows per 256-byte bank window
constexpr int ROWS_PER_PIECE = 512 / BK;    // rows per 1 KB DMA piece
constexpr int PIECES = BM * BK / 512;       // 1 KB pieces per operand stage
constexpr int PPW = PIECES / kWaves;        // pieces per wave per operand
constexpr int kStage = BM * BK;             // elements per operand stage
// Split-K of the last, partial round of tiles: at most kMaxSplit pieces per
// tile, each at least kMinSplitSteps K-steps; a piece's fp32 partial tile is
// 256 threads x 64 float4 (256 KB) in the workspace. A piece pays a prologue,
// its partial tile's stores and a share of the final sum whatever its length,
// which shorter pieces do not earn back: with K = 2048 (64 steps) four
// 16-step pieces made the launch slower than no split at all.
constexpr int kMaxSplit = 8, kMinSplitSteps = 64;
constexpr int kMaxPieces = 512;
constexpr size_t kPieceBytes = 256 * 64 * 16;
static_assert(BM == BN, "A and B stages share the piece layout");
static_assert(STAGES * 2 * kStage * 2 <= 160 * 1024, "LDS");
static_assert(STAGES == 4 || STAGES == 5, "the K loop is written for four or five stages");
__device__ __forceinline__ int swz(int r, int c) { return c ^ ((r / RPW) % CPR); }
}  // namespace fast

// The fast path addresses one expert's weight matrix, and 256 rows of an
// activation, with 32-bit byte offsets.
inline bool fast_path(int64_t H, int64_t F) {
  return H % fast::BK == 0 && F % fast::BK == 0 && F * H < ((int64_t)1 << 31);
}

// Partial tiles the workspace holds for the split tail of either GEMM.
inline int64_t max_split_pieces(int64_t max_rows, int64_t H, int64_t F, int E) {
  const int64_t row_tiles = ceil_div(max_rows, fast::BM) + E;
  const int64_t col_tiles = std::max(ceil_div(F, fast::BN / 2), ceil_div(H, fast::BN));
  return std::min<int64_t>(fast::kMaxPieces,
                           fast::kMaxSplit * std::min<int64_t>(row_tiles * col_tiles, kMaxTailTiles));
}

// Workgroup barrier for the K loop: this wave's LDS reads have returned
// (a stage is refilled by DMA only after every wave passed the barrier that
// follows its last reads) and its DMA of the awaited step was waited for
// beforehand; no memory fence, which would drain every DMA in flight. The
// asm's memory clobber keeps the compiler from moving any load or store
// (LDS reads of the next stage in particular) across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int EPI>
__global__ void __launch_bounds__(fast::kThreads, 1)
ffn_gemm_bf16_fast(const uint16_t* __restrict__ A, int64_t K,
                 const uint16_t* __restrict__ B0, const uint16_t* __restrict__ B1,
                 int64_t F, int64_t H,
                 const int32_t* __restrict__ offsets, const int32_t* __restrict__ slot,
                 int E, int64_t max_rows, const int32_t* __restrict__ prefix,
                 const int32_t* __restrict__ prefix2,
                 int32_t* __restrict__ claim, int32_t* __restrict__ tail,
                 float* __restrict__ partial, int max_pieces, uint16_t* __restrict__ C) {
  constexpr int BM = fast::BM, BN = fast::BN, BK = fast::BK, STAGES = fast::STAGES;
  constexpr int CPR = fast::CPR, ROWS_PER_PIECE = fast::ROWS_PER_PIECE, PPW = fast::PPW;
  constexpr int kStage = fast::kStage;
  auto swz = [](int r, int c) { return fast::swz(r, c); };
  constexpr int kOutN = EPI == 0 ? BN / 2 : BN;
  const int64_t N_out = EPI == 0 ? F : H;
  const int64_t ldc = N_out;
  const int64_t n_tiles = (N_out + kOutN - 1) / kOutN;

  constexpr int kStage4 = STAGES > 4 ? kStage : 8;   // a fifth stage, or only the claim words
  __shared__ __attribute__((aligned(1024))) uint16_t As0[kStage], As1[kStage], As2[kStage], As3[kStage];
  __shared__ __attribute__((aligned(1024))) uint16_t Bs0[kStage], Bs1[kStage], Bs2[kStage], Bs3[kStage];
  __shared__ __attribute__((aligned(1024))) uint16_t As4[kStage4];
  __shared__ __attribute__((aligned(1024))) uint16_t Bs4[STAGES > 4 ? kStage : 1];
  uint16_t* const As[5] = {As0, As1, As2, As3, As4};
  uint16_t* const Bs[5] = {Bs0, Bs1, Bs2, Bs3, Bs4};
  // The claim broadcast lives in the fifth A stage: it is written and read
  // between tiles, when no DMA targets that stage (a tile's first STAGES - 1
  // steps load stages 0 .. STAGES - 2), and s_last after every wave has left
  // the K loop.
  int64_t& s_claim = *reinterpret_cast<int64_t*>(As4);
  int& s_piece = *reinterpret_cast<int*>(As4 + 4);
  int& s_last = *reinterpret_cast<int*>(As4 + 6);

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int frow = lane & 31;                 // fragment row within a 32-row MFMA tile
  const int fk = lane >> 5;                   // which 8-wide half of a 16-wide K step
  const int lrow = lane / CPR;                // row within a DMA piece
  const int lpch = lane % CPR;                // physical chunk this lane fills

  // tiles: every expert's full-cost row tiles (prefix), then the small last
  // row tiles (prefix2), each in (expert, column tile, row tile) order
  const int64_t total_big = (int64_t)prefix[E] * n_tiles;
  const int64_t total = total_big + (int64_t)prefix2[E] * n_tiles;
  if (total == 0) return;                      // every expert went to the few-row kernels
  const int64_t G = gridDim.x;                 // persistent grid, a multiple of 8
  const int64_t per_xcd = G / 8;
  // Claim chunk: an XCD's whole share of a round, or 16 consecutive tiles
  // when some expert has 8 or more full-cost row tiles (a column's row tiles
  // then fill a 32-tile chunk by themselves, one weight tile against 32
  // activation panels; 16 divides the share, so the chunks of the 8 XCDs
  // still cover each round exactly once). With at most 7 row tiles per expert
  // the larger chunk cuts fewer column groups across two XCDs' L2s.
  int64_t me_max = 0;
  for (int ee = 0; ee < E; ++ee) me_max = max(me_max, (int64_t)(prefix[ee + 1] - prefix[ee]));
  const int64_t chunk = me_max >= 8 && per_xcd % 16 == 0 ? 16 : per_xcd;
  const int xcd = blockIdx.x % 8;
  const int64_t ksteps = K / BK;

  // Whole rounds of G tiles are claimed per XCD (each XCD walks its own
  // chunks of consecutive tiles, so the row tiles that share a weight tile
  // run together on one L2). The last, partial round of rem tiles is
  // split along K into `split` pieces claimed from one global counter,
  // chosen to minimise ceil(rem * split / G) / split rounds.
  const int64_t full = total / G * G;
  const int64_t rem = total - full;
  int64_t split = 1;
  for (int64_t sp = 2; sp <= fast::kMaxSplit; ++sp) {
    if (ksteps / sp < fast::kMinSplitSteps || rem * sp > max_pieces) break;
    if (((rem * sp + G - 1) / G) * split < ((rem * split + G - 1) / G) * sp) split = sp;
  }

  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  using I4 = std::integral_constant<int, 4>;

  bool in_tail = false;                        // thread 0 only
  // thread 0: the next whole-round claim, issued while the current tile runs
  // The counter's address is made opaque so the compiler does not rewrite the
  // one-lane atomic into its wave-aggregated form, which reads the result at
  // once; this way the round trip overlaps the tile and only the next claim
  // waits for it.
  __attribute__((address_space(1))) int32_t* claim_x =
      (__attribute__((address_space(1))) int32_t*)(claim + xcd);
  asm volatile("" : "+v"(claim_x));
  int32_t j_next =
      tid == 0 ? __hip_atomic_fetch_add(claim_x, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
  for (;;) {
    if (tid == 0) {
      int64_t tt = -1;
      int pc = 0;
      if (!in_tail) {
        const int64_t j = j_next;
        const int64_t c = ((j / chunk) * 8 + xcd) * chunk + (j % chunk);
        if (c < full) tt = c;
        else in_tail = true;
      }
      if (in_tail) {
        const int64_t u = atomicAdd(&tail[0], 1);
        if (u < rem * split) {
          tt = full + u / split;
          pc = (int)(u % split);
        }
      }
      s_claim = tt;
      s_piece = pc;
    }
    // LDS only: the claim, and every wave's last reads of the staging stages
    // before the prologue refills them; the previous epilogue's global
    // stores drain on their own (nothing in this launch reads them)
    lds_barrier();
    const int64_t t = s_claim;
    const int piece = s_piece;
    if (t < 0) break;
    if (tid == 0 && !in_tail)
      j_next = __hip_atomic_fetch_add(claim_x, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const bool split_tile = t >= full && split > 1;
    const int64_t kbeg = split_tile ? piece * ksteps / split : 0;
    const int64_t nks = split_tile ? (piece + 1) * ksteps / split - kbeg : ksteps;
    // the last expert whose first tile is at or before t (binary search)
    int e = 0;
    int64_t nt, mt;
    if (t < total_big) {
      for (int hi = E - 1; e < hi;) {
        const int mid = (e + hi + 1) >> 1;
        if ((int64_t)prefix[mid] * n_tiles <= t) e = mid;
        else hi = mid - 1;
      }
      const int64_t local = t - (int64_t)prefix[e] * n_tiles;
      const int64_t me = prefix[e + 1] - prefix[e];
      nt = local / me;
      mt = local - nt * me;
    } else {
      const int64_t u = t - total_big;
      const int64_t si = u / n_tiles;          // which small row tile
      for (int hi = E - 1; e < hi;) {
        const int mid = (e + hi + 1) >> 1;
        if ((int64_t)prefix2[mid] <= si) e = mid;
        else hi = mid - 1;
      }
      nt = u - si * n_tiles;
      mt = prefix[e + 1] - prefix[e];          // after the expert's full-cost tiles
    }
    const int s = slot ? slot[e] : e;
    int64_t lo = offsets[e];
    lo = lo < 0 ? 0 : (lo > max_rows ? max_rows : lo);
    int64_t hi = offsets[e + 1];
    hi = hi < lo ? lo : (hi > max_rows ? max_rows : hi);
    const int64_t row0 = lo + mt * BM;
    const int64_t row_end = min(row0 + (int64_t)BM, hi);
    const int64_t n0 = nt * kOutN;
    const int nrows = (int)(row_end - row0);

    // DMA sources: a wave-uniform base per piece plus a 32-bit byte offset
    // per lane (the K offset is added to the base per step). Rows past the
    // end of the expert or of the weight read a valid row; their results are
    // never stored. Inside the K loop the stepped base and the lane offset
    // pass through empty asm, so the load takes the scalar-base form (SGPR
    // pair + 32-bit VGPR offset) and the K step costs scalar adds, rather than
    // 64-bit per-lane pointers stepped with vector adds.
    const char* const a_base = reinterpret_cast<const char*>(A + row0 * K);
    const char* b_base[PPW];
    uint32_t a_off[PPW], b_off[PPW];
#pragma unroll
    for (int i = 0; i < PPW; ++i) {
      const int piece = wave * PPW + i;
      const int r = piece * ROWS_PER_PIECE + lrow;
      const int lch = swz(r, lpch);
      a_off[i] = (uint32_t)(((r < nrows ? r : 0) * K + lch * 8) * 2);
      int64_t wrow;
      if (EPI == 0) {
        const int grp = piece >> 1;              // 32-row groups: gate, up, gate, up, ...
        int64_t f = n0 + (grp >> 1) * 32 + (r & 31);
        if (f >= F) f = 0;
        b_base[i] = reinterpret_cast<const char*>(((grp & 1) ? B1 : B0) + (int64_t)s * F * H);
        wrow = f;
      } else {
        int64_t h = n0 + r;
        if (h >= H) h = 0;
        b_base[i] = reinterpret_cast<const char*>(B0 + (int64_t)s * H * F);
        wrow = h;
      }
      b_off[i] = (uint32_t)((wrow * K + lch * 8) * 2);
    }
    auto issue = [&](auto stage_c, int64_t step) {
      constexpr int stage = decltype(stage_c)::value;
      const int64_t kb = (kbeg + step) * BK * 2;
#pragma unroll
      for (int i = 0; i < PPW; ++i) {
        const char* ab = a_base + kb;
        const char* bb = b_base[i] + kb;
        uint32_t ao = a_off[i], bo = b_off[i];
        asm("" : "+s"(ab), "+s"(bb), "+v"(ao), "+v"(bo));
        lds_dma16(ab + ao, As[stage] + (wave * PPW + i) * 512);
        lds_dma16(bb + bo, Bs[stage] + (wave * PPW + i) * 512);
      }
    };
    auto issue_a = [&](auto stage_c, int64_t step) {
      constexpr int stage = decltype(stage_c)::value;
      const int64_t kb = (kbeg + step) * BK * 2;
      const char* ab = a_base + kb;
      asm("" : "+s"(ab));
#pragma unroll
      for (int i = 0; i < PPW; ++i) {
        uint32_t ao = a_off[i];
        asm("" : "+v"(ao));
        lds_dma16(ab + ao, As[stage] + (wave * PPW + i) * 512);
      }
    };
    auto issue_b = [&](auto stage_c, int64_t step) {
      constexpr int stage = decltype(stage_c)::value;
      const int64_t kb = (kbeg + step) * BK * 2;
#pragma unroll
      for (int i = 0; i < PPW; ++i) {
        const char* bb = b_base[i] + kb;
        uint32_t bo = b_off[i];
        asm("" : "+s"(bb), "+v"(bo));
        lds_dma16(bb + bo, Bs[stage] + (wave * PPW + i) * 512);
      }
    };

    // MODE 0: 2 x 2 waves of 128 x 128; MODE m in {1, 2, 4}: 4 waves side by
    // side, each m x 32 rows by 64 columns.
    auto run = [&](auto mode_c) {
      constexpr int MODE = decltype(mode_c)::value;
      constexpr bool FULL = MODE == 0;
      constexpr int MI = FULL ? 4 : MODE;
      constexpr int NI = FULL ? 4 : 2;
      const int rbase = FULL ? (wave >> 1) * 128 : 0;
      const int cbase = FULL ? (wave & 1) * 128 : wave * 64;

      f32x16_t acc[MI][NI];
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
#pragma unroll
          for (int q = 0; q < 16; ++q) acc[mi][ni][q] = 0.f;
      bf16x8_t fa0[MI], fb0[NI], fa1[MI], fb1[NI];

      auto rd = [&](auto stage_c, int ks, bf16x8_t (&fa)[MI], bf16x8_t (&fb)[NI]) {
        constexpr int J = decltype(stage_c)::value;
        const uint16_t* as = As[J];
        const uint16_t* bs = Bs[J];
        const int ch = ks * 2 + fk;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
          const int r = rbase + mi * 32 + frow;
          fa[mi] = *reinterpret_cast<const bf16x8_t*>(&as[r * BK + swz(r, ch) * 8]);
        }
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) {
          const int r = cbase + ni * 32 + frow;
          fb[ni] = *reinterpret_cast<const bf16x8_t*>(&bs[r * BK + swz(r, ch) * 8]);
        }
      };
      auto mm = [&](const bf16x8_t (&fa)[MI], const bf16x8_t (&fb)[NI]) {
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
#pragma unroll
          for (int ni = 0; ni < NI; ++ni)
            acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[mi], fb[ni], acc[mi][ni], 0, 0, 0);
      };
      // Wait until at most n steps issued after the awaited one are in flight.
      auto wait_steps = [&](int64_t n) {
        if constexpr (STAGES >= 5) {
          if (n >= 3) {
            wait_vmcnt<3 * 2 * PPW>();
            return;
          }
        }
        if (n >= 2) wait_vmcnt<2 * 2 * PPW>();
        else if (n == 1) wait_vmcnt<2 * PPW>();
        else wait_vmcnt<0>();
      };
      // One K-step on stage J: DMA of step kt+3 into stage J+3 (mod 4); the
      // second half-step's fragments are read while the first half's MFMAs
      // run; wait for step kt+1; barrier; the next step's first fragments are
      // read while this step's second half runs.
      auto step = [&](auto j_c, int64_t kt) {
        constexpr int J = decltype(j_c)::value;
        if (kt + STAGES - 1 < nks)
          issue(std::integral_constant<int, (J + STAGES - 1) % STAGES>{}, kt + STAGES - 1);
        rd(j_c, 1, fa1, fb1);
        mm(fa0, fb0);
        wait_steps(min(kt + STAGES - 1, nks - 1) - (kt + 1));
        lds_barrier();
        if (kt + 1 < nks) rd(std::integral_constant<int, (J + 1) % STAGES>{}, 0, fa0, fb0);
        mm(fa1, fb1);
      };

      // Steady state (steps kt + 3 < nks): the same step with every
      // condition known, so the waits are fixed and exact.
      auto step_ss = [&](auto j_c, int64_t kt) {
        constexpr int J = decltype(j_c)::value;
        constexpr int JN = (J + STAGES - 1) % STAGES;
        issue_a(std::integral_constant<int, JN>{}, kt + STAGES - 1);
        rd(j_c, 1, fa1, fb1);
        mm(fa0, fb0);
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        }
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        }
        // outstanding after step kt+1: A and B of steps kt+2 .. kt+STAGES-2,
        // A of kt+STAGES-1
        wait_vmcnt<(2 * (STAGES - 3) + 1) * PPW>();
        lds_barrier();
        issue_b(std::integral_constant<int, JN>{}, kt + STAGES - 1);
        rd(std::integral_constant<int, (J + 1) % STAGES>{}, 0, fa0, fb0);
        mm(fa1, fb1);
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 1);
        }
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
          __builtin_amdgcn_sched_group_barrier(0x020, 1, 1);
          __builtin_amdgcn_sched_group_barrier(0x008, 2, 1);
        }
      };

      if (0 < nks) issue(I0{}, 0);
      if (1 < nks) issue(I1{}, 1);
      if (2 < nks) issue(I2{}, 2);
      if constexpr (STAGES >= 5)
        if (3 < nks) issue(I3{}, 3);
      wait_steps(min((int64_t)STAGES - 1, nks) - 1);
      // every wave has its own pieces of step 0; the barrier makes that true
      // of all of them (LDS only: steps 1 and 2 keep loading)
      lds_barrier();
      rd(I0{}, 0, fa0, fb0);
      int64_t kt = 0;
      for (; kt + STAGES + STAGES - 1 <= nks; kt += STAGES) {
        step_ss(I0{}, kt);
        step_ss(I1{}, kt + 1);
        step_ss(I2{}, kt + 2);
        step_ss(I3{}, kt + 3);
        if constexpr (STAGES >= 5) step_ss(I4{}, kt + 4);
      }
      for (; kt + STAGES <= nks; kt += STAGES) {
        step(I0{}, kt);
        step(I1{}, kt + 1);
        step(I2{}, kt + 2);
        step(I3{}, kt + 3);
        if constexpr (STAGES >= 5) step(I4{}, kt + 4);
      }
      if (kt < nks) step(I0{}, kt);
      if (kt + 1 < nks) step(I1{}, kt + 1);
      if (kt + 2 < nks) step(I2{}, kt + 2);
      if constexpr (STAGES >= 5)
        if (kt + 3 < nks) step(I3{}, kt + 3);

      // A K-piece stores its fp32 partial tile; the piece that arrives last
      // (a device-scope counter per tail tile, ordered by release and acquire
      // fences) adds all pieces in piece order, so the sum does not depend on
      // arrival order, and writes the output.
      if (split_tile) {
        constexpr int kF4 = fast::kPieceBytes / 16 / 256;       // float4 per thread
        static_assert(MI * NI * 4 <= kF4, "partial tile layout");
        const int64_t tile_slot = t - full;
        f32x4_t* const P = reinterpret_cast<f32x4_t*>(partial);
        f32x4_t* const mine = P + (tile_slot * split + piece) * (int64_t)kF4 * 256;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
#pragma unroll
          for (int ni = 0; ni < NI; ++ni)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
              f32x4_t v;
              v[0] = acc[mi][ni][4 * q4];
              v[1] = acc[mi][ni][4 * q4 + 1];
              v[2] = acc[mi][ni][4 * q4 + 2];
              v[3] = acc[mi][ni][4 * q4 + 3];
              mine[((mi * NI + ni) * 4 + q4) * 256 + tid] = v;
            }
        __threadfence();
        __syncthreads();
        if (tid == 0) s_last = atomicAdd(&tail[1 + tile_slot], 1) == (int)split - 1;
        __syncthreads();
        if (!s_last) return;
        __threadfence();
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
#pragma unroll
          for (int ni = 0; ni < NI; ++ni)
#pragma unroll
            for (int q = 0; q < 16; ++q) acc[mi][ni][q] = 0.f;
        for (int64_t pc = 0; pc < split; ++pc) {
          const f32x4_t* const src = P + (tile_slot * split + pc) * (int64_t)kF4 * 256;
#pragma unroll
          for (int mi = 0; mi < MI; ++mi)
#pragma unroll
            for (int ni = 0; ni < NI; ++ni)
#pragma unroll
              for (int q4 = 0; q4 < 4; ++q4) {
                const f32x4_t v = src[((mi * NI + ni) * 4 + q4) * 256 + tid];
                acc[mi][ni][4 * q4] += v[0];
                acc[mi][ni][4 * q4 + 1] += v[1];
                acc[mi][ni][4 * q4 + 2] += v[2];
                acc[mi][ni][4 * q4 + 3] += v[3];
              }
        }
      }

      // Epilogue, staged through LDS (the stages are free: every wave passed
      // the last K-step's barrier after its last fragment read). Each wave
      // writes its bf16 results into the tile, 32 rows per stage array, with
      // the 16-byte chunks of a row XOR-swizzled by (row mod 8); then the
      // block stores whole rows with 16-byte coalesced writes.
      // 32x32 C layout: column lane % 32, rows 8*(q/4) + 4*(lane/32) + q%4.
      constexpr int NOUT = kOutN;                       // output columns of the tile
      // Stage array holding rows [32 b, 32 b + 32) of the tile (b compile-time).
      auto stage_of = [&](auto b_c) -> uint16_t* {
        constexpr int b = decltype(b_c)::value;
        if constexpr (b < 4) return As[b];
        else return Bs[b - 4];
      };
      auto off_in = [](int r, int c) {               // r: row within the 32-row block
        return r * NOUT + ((((c >> 3) ^ (r & 7)) << 3) | (c & 7));
      };
      // Lane coordinates are made opaque per tile so that the write addresses
      // derived from them are formed here, not hoisted out of the tile loop.
      int ccol = lane & 31;
      int crow = (lane >> 5) * 4;
      asm volatile("" : "+v"(ccol), "+v"(crow));
      // wave's rows: 32-row blocks (rbase / 32) + mi
      auto write_rows = [&](auto b0_c) {
        constexpr int B0 = decltype(b0_c)::value;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
          uint16_t* const base = mi == 0 ? stage_of(std::integral_constant<int, B0>{})
                               : mi == 1 ? stage_of(std::integral_constant<int, B0 + 1>{})
                               : mi == 2 ? stage_of(std::integral_constant<int, (B0 + 2) % 8>{})
                                         : stage_of(std::integral_constant<int, (B0 + 3) % 8>{});
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            const int r = 8 * (q >> 2) + crow + (q & 3);
            if (EPI == 0) {
#pragma unroll
              for (int p = 0; p < NI / 2; ++p) {
                const float g = acc[mi][2 * p][q];
                const float u = acc[mi][2 * p + 1][q];
                base[off_in(r, cbase / 2 + p * 32 + ccol)] = f32_to_bf16(swiglu(g, u));
              }
            } else {
#pragma unroll
              for (int ni = 0; ni < NI; ++ni)
                base[off_in(r, cbase + ni * 32 + ccol)] = f32_to_bf16(acc[mi][ni][q]);
            }
          }
        }
      };
      if (FULL && (wave >> 1)) write_rows(std::integral_constant<int, 4>{});
      else write_rows(std::integral_constant<int, 0>{});
      __syncthreads();
      // Rows of the tile that hold results: all 256 in a full tile, MI * 32
      // when the waves sit side by side.
      constexpr int CPRO = NOUT / 8;                    // 16-byte chunks per output row
      const int rows_here = min(nrows, FULL ? BM : MI * 32);
      int64_t ld = ldc;
      asm volatile("" : "+s"(ld));
      int tid_o = tid;
      asm volatile("" : "+v"(tid_o));
      auto store_block = [&](auto b_c) {
        constexpr int b = decltype(b_c)::value;
        const uint16_t* const base = stage_of(b_c);
#pragma unroll
        for (int qd0 = 0; qd0 < 32 * CPRO; qd0 += fast::kThreads) {
          const int qd = qd0 + tid_o;
          const int r = qd / CPRO, ch = qd - r * CPRO;
          if (b * 32 + r < rows_here && n0 + ch * 8 < N_out) {
            const uint4 v = *reinterpret_cast<const uint4*>(base + off_in(r, ch * 8));
            *reinterpret_cast<uint4*>(C + (row0 + b * 32 + r) * ld + n0 + ch * 8) = v;
          }
        }
      };
      store_block(std::integral_constant<int, 0>{});
      store_block(std::integral_constant<int, 1>{});
      store_block(std::integral_constant<int, 2>{});
      store_block(std::integral_constant<int, 3>{});
      if (FULL) {
        store_block(std::integral_constant<int, 4>{});
        store_block(std::integral_constant<int, 5>{});
        store_block(std::integral_constant<int, 6>{});
        store_block(std::integral_constant<int, 7>{});
      }
    };
    if (nrows > 128) run(std::integral_constant<int, 0>{});
    else if (nrows > 64) run(std::integral_constant<int, 4>{});
    else if (nrows > 32) run(std::integral_constant<int, 2>{});
    else run(std::integral_constant<int, 1>{});
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
  using namespace moe;
  if (max_rows < 1 || H < 1 || F < 1 || E < 1 || !valid_dtype(dtype)) return 0;
  const size_t elt = dtype == MOE_BF16 ? 2 : 4;
  size_t bytes = align_up((size_t)max_rows * (size_t)F * elt, 256);
  bytes += align_up((size_t)(E + 1 + kCounterWords + 2 * (E + 1)) * sizeof(int32_t), 256);
  if (dtype == MOE_BF16 && fast_path(H, F))
    bytes += (size_t)max_split_pieces(max_rows, H, F, E) * fast::kPieceBytes;
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

  const bool fast = fast_path(H, F);
  const int bm = fast ? fast::BM : BM;
  // Experts with at most 16 * kSmallMaxTiles rows go to the weight-streaming
  // kernel when the batch is decode-sized (at most 64 rows per expert on
  // average): bf16, H and F multiples of 32 (the fast-path shapes), 32-bit lane
  // offsets within 96 rows of K. Larger batches leave the rare small expert to
  // the large tiles and launch no few-row kernel at all.
  const int small_tiles =
      fast && std::max(H, F) < ((int64_t)1 << 24) && max_rows <= 64 * (int64_t)E ? kSmallMaxTiles : 0;
  ffn_tiles_kernel<<<dim3(1), dim3(64), 0, st>>>(expert_offsets, slot_of_expert, E, S, max_rows,
                                                 bm, small_tiles, fast ? 1 : 0, prefix);
  MOE_CHECK_LAUNCH();
  const int32_t* const small = prefix + E + 1 + kCounterWords;
  const int32_t* const prefix2 = small + E + 1;
  const bool few = small_tiles > 0;
  const bool big = max_rows > 16 * small_tiles;  // else every expert has few rows
  // the most row tiles a listed expert can have, rounded up to a compiled bound
  const int64_t few_tiles = std::min<int64_t>(ceil_div(max_rows, 16), small_tiles);
  const int mtmax = few_tiles <= 1 ? 1 : few_tiles <= 2 ? 2 : few_tiles <= 4 ? 4 : 6;
  int grid = device_cu_count();
  grid = std::min((grid + 7) / 8 * 8, kMaxTailTiles);     // a tail round has < grid tiles
  const auto* xb = static_cast<const uint16_t*>(x_perm);
  auto* ab = static_cast<uint16_t*>(act);
  const auto* wgb = static_cast<const uint16_t*>(w_gate);
  const auto* wub = static_cast<const uint16_t*>(w_up);
  const auto* wdb = static_cast<const uint16_t*>(w_down);
  auto* yb = static_cast<uint16_t*>(y_perm);
  if (fast) {
    int32_t* const claim = prefix + E + 1;
    int32_t* const tail = claim + kClaimWords;
    float* const partial = reinterpret_cast<float*>(
        reinterpret_cast<char*>(prefix) + align_up((size_t)(E + 1 + kCounterWords + 2 * (E + 1)) * 4, 256));
    const int pieces = (int)max_split_pieces(max_rows, H, F, E);
    // two blocks per compute unit, striding over the few-row experts' units
    // (more blocks in flight spread the reads over more DRAM rows at once and
    // measured slower; fewer leave bandwidth unused); with few units each
    // block does one
    auto small_grid = [&](int64_t n_out, int cols) {
      return (unsigned)std::min<int64_t>(2 * (int64_t)device_cu_count(), (int64_t)E * ceil_div(n_out, cols));
    };
    auto launch_small = [&](auto epi_c, const uint16_t* a, int64_t K, const uint16_t* b0,
                            const uint16_t* b1, uint16_t* c) {
      constexpr int EPI = decltype(epi_c)::value;
      const unsigned g = small_grid(EPI == 0 ? F : H, SmallShape<EPI>::COLS);
      const dim3 blk(64 * kSmallWaves);
      if (mtmax == 1)
        ffn_small_bf16<EPI, 1><<<dim3(g), blk, 0, st>>>(a, K, b0, b1, F, H, expert_offsets,
                                                        slot_of_expert, max_rows, small, c);
      else if (mtmax == 2)
        ffn_small_bf16<EPI, 2><<<dim3(g), blk, 0, st>>>(a, K, b0, b1, F, H, expert_offsets,
                                                        slot_of_expert, max_rows, small, c);
      else if (mtmax == 4)
        ffn_small_bf16<EPI, 4><<<dim3(g), blk, 0, st>>>(a, K, b0, b1, F, H, expert_offsets,
                                                        slot_of_expert, max_rows, small, c);
      else
        ffn_small_bf16<EPI, 6><<<dim3(g), blk, 0, st>>>(a, K, b0, b1, F, H, expert_offsets,
                                                        slot_of_expert, max_rows, small, c);
    };
    if (big) {
      ffn_gemm_bf16_fast<0><<<dim3(grid), dim3(fast::kThreads), 0, st>>>(
          xb, H, wgb, wub, F, H, expert_offsets, slot_of_expert, E, max_rows, prefix,
          prefix2, claim, tail, partial, pieces, ab);
      MOE_CHECK_LAUNCH();
    }
    if (few) {
      launch_small(std::integral_constant<int, 0>{}, xb, H, wgb, wub, ab);
      MOE_CHECK_LAUNCH();
    }
    if (big) {
      ffn_gemm_bf16_fast<1><<<dim3(grid), dim3(fast::kThreads), 0, st>>>(
          ab, F, wdb, nullptr, F, H, expert_offsets, slot_of_expert, E, max_rows, prefix,
          prefix2, claim + 8, tail + kTailWords, partial, pieces, yb);
      MOE_CHECK_LAUNCH();
    }
    if (few) {
      launch_small(std::integral_constant<int, 1>{}, ab, F, wdb, nullptr, yb);
      MOE_CHECK_LAUNCH();
    }
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
