// moe_permute: stable expert-major grouping of (token, choice) pairs and the
// gather of hidden-state rows into that order.
//
// Four launches, all on the caller's stream:
//   1. count   -- each block counts the experts of a contiguous chunk of pairs
//                 in an LDS histogram;
//   2. scan    -- one block turns the per-chunk counts into expert offsets and
//                 per-(chunk, expert) starting rows (exclusive scans);
//   3. rank    -- each block walks its chunk again in pair order; inside a
//                 wavefront, lanes holding the same expert are found with eight
//                 ballots (one per bit of the id), so a pair's stable rank is a
//                 popcount of the lower lanes in its match mask; wave totals
//                 are carried across the block through LDS;
//   4. gather  -- one wavefront per batch token reads the token's row once with
//                 16-byte loads and writes it to each of its k destination rows.
#include "common.h"

namespace moe {
namespace {

constexpr int kPermThreads = 256;
constexpr int kPermChunk = 4096;   // pairs per block in count/rank

struct PairSrc {
  const int32_t* token_ids;
  const int32_t* idx;
  int64_t n_tokens;
  int k;
  int E;
};

// Expert of pair p, or -1 when the pair's token or expert id is out of range.
__device__ __forceinline__ int pair_expert(const PairSrc& s, int64_t p) {
  const int64_t i = p / s.k;
  const int j = (int)(p - i * s.k);
  const int64_t t = s.token_ids ? (int64_t)s.token_ids[i] : i;
  if (t < 0 || t >= s.n_tokens) return -1;
  const int e = s.idx[t * s.k + j];
  return (e >= 0 && e < s.E) ? e : -1;
}

__global__ void __launch_bounds__(kPermThreads)
perm_count_kernel(PairSrc src, int64_t P, int32_t* __restrict__ counts) {
  __shared__ int32_t hist[256];
  for (int e = threadIdx.x; e < src.E; e += blockDim.x) hist[e] = 0;
  __syncthreads();
  const int64_t start = (int64_t)blockIdx.x * kPermChunk;
  const int64_t end = min(start + (int64_t)kPermChunk, P);
  for (int64_t p = start + threadIdx.x; p < end; p += blockDim.x) {
    const int e = pair_expert(src, p);
    if (e >= 0) atomicAdd(&hist[e], 1);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < src.E; e += blockDim.x)
    counts[(int64_t)blockIdx.x * src.E + e] = hist[e];
}

// One block of 256 threads; thread e owns expert e.
__global__ void __launch_bounds__(256)
perm_scan_kernel(const int32_t* __restrict__ counts, int64_t nblk, int E,
                 int32_t* __restrict__ bases, int32_t* __restrict__ offsets) {
  __shared__ int32_t tot[256];
  const int e = threadIdx.x;
  int32_t total = 0;
  if (e < E)
    for (int64_t b = 0; b < nblk; ++b) total += counts[b * E + e];
  tot[e] = (e < E) ? total : 0;
  __syncthreads();
  // Exclusive scan over experts (E <= 256; a serial pass by one wave lane is
  // cheap and keeps the order obvious).
  __shared__ int32_t off[257];
  if (threadIdx.x == 0) {
    int32_t run = 0;
    for (int q = 0; q < E; ++q) {
      off[q] = run;
      run += tot[q];
    }
    off[E] = run;
  }
  __syncthreads();
  if (e < E) {
    offsets[e] = off[e];
    int32_t run = off[e];
    for (int64_t b = 0; b < nblk; ++b) {
      bases[b * E + e] = run;
      run += counts[b * E + e];
    }
  }
  if (threadIdx.x == 0) offsets[E] = off[E];
}

__global__ void __launch_bounds__(kPermThreads)
perm_rank_kernel(PairSrc src, int64_t P, const int32_t* __restrict__ bases,
                 int32_t* __restrict__ row_of_pair, int32_t* __restrict__ pair_of_row) {
  constexpr int kWaves = kPermThreads / kWave;
  __shared__ int32_t running[256];
  __shared__ int32_t wave_cnt[kWaves][256];
  const int wave = threadIdx.x / kWave;
  for (int e = threadIdx.x; e < src.E; e += blockDim.x) {
    running[e] = 0;
    for (int w = 0; w < kWaves; ++w) wave_cnt[w][e] = 0;
  }
  __syncthreads();
  const int64_t start = (int64_t)blockIdx.x * kPermChunk;
  const int64_t end = min(start + (int64_t)kPermChunk, P);
  const int32_t* base = bases + (int64_t)blockIdx.x * src.E;
  for (int64_t r0 = start; r0 < end; r0 += kPermThreads) {
    const int64_t p = r0 + threadIdx.x;
    const int e = (p < end) ? pair_expert(src, p) : -1;
    const bool valid = e >= 0;
    // Lanes of this wave holding the same expert id: intersect, bit by bit,
    // the ballots that agree with this lane's id.
    uint64_t match = ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const bool b = valid && ((e >> bit) & 1);
      const uint64_t bal = ballot(b);
      match &= b ? bal : ~bal;
    }
    const int rank_in_wave = __popcll(match & lanemask_lt());
    if (valid && (match & lanemask_lt()) == 0) wave_cnt[wave][e] = __popcll(match);
    __syncthreads();
    if (valid) {
      int32_t before = running[e];
      for (int w = 0; w < wave; ++w) before += wave_cnt[w][e];
      const int32_t row = base[e] + before + rank_in_wave;
      row_of_pair[p] = row;
      pair_of_row[row] = (int32_t)p;
    } else if (p < end) {
      row_of_pair[p] = -1;
    }
    __syncthreads();
    for (int q = threadIdx.x; q < src.E; q += blockDim.x) {
      int32_t add = 0;
      for (int w = 0; w < kWaves; ++w) {
        add += wave_cnt[w][q];
        wave_cnt[w][q] = 0;
      }
      running[q] += add;
    }
    __syncthreads();
  }
}

// Rows are moved as 16-byte vectors; row_vecs = row bytes / 16.
__global__ void __launch_bounds__(256)
perm_gather_kernel(const uint4* __restrict__ x, const int32_t* __restrict__ token_ids,
                   int64_t T, int64_t n_tokens, int k, int64_t row_vecs,
                   const int32_t* __restrict__ row_of_pair, int64_t P,
                   uint4* __restrict__ x_perm) {
  const int64_t i = (int64_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
  if (i >= T) return;
  const int64_t t = token_ids ? (int64_t)token_ids[i] : i;
  if (t < 0 || t >= n_tokens) return;
  const uint4* src = x + t * row_vecs;
  const int32_t* rows = row_of_pair + i * k;
  for (int64_t c = lane_id(); c < row_vecs; c += kWave) {
    const uint4 v = src[c];
    for (int j = 0; j < k; ++j) {
      const int32_t r = rows[j];
      if (r >= 0 && r < P) x_perm[(int64_t)r * row_vecs + c] = v;
    }
  }
}

}  // namespace
}  // namespace moe

extern "C" size_t moe_permute_workspace(int64_t T, int32_t k, int32_t E) {
  if (T < 1 || k < 1 || E < 1) return 0;
  const int64_t nblk = moe::ceil_div(T * k, moe::kPermChunk);
  return moe::align_up((size_t)(2 * nblk * E) * sizeof(int32_t), 256);
}

extern "C" int moe_permute(const void* x, int32_t dtype, int64_t H, int64_t n_tokens,
                           const int32_t* token_ids, int64_t T, const int32_t* topk_idx,
                           int32_t k, int32_t E, int32_t* expert_offsets,
                           int32_t* row_of_pair, int32_t* pair_of_row, void* x_perm,
                           void* workspace, size_t ws_bytes, void* stream) {
  using namespace moe;
  MOE_CHECK_ARG(T >= 1 && k >= 1 && E >= 1 && E <= 256 && k <= E);
  MOE_CHECK_ARG(n_tokens >= 1 && (token_ids != nullptr || n_tokens >= T));
  MOE_CHECK_ARG(topk_idx && expert_offsets && row_of_pair && pair_of_row);
  MOE_CHECK_ARG((x == nullptr) == (x_perm == nullptr));
  const int64_t P = T * (int64_t)k;
  MOE_CHECK_ARG(P < ((int64_t)1 << 31));
  int64_t row_vecs = 0;
  if (x) {
    MOE_CHECK_ARG(valid_dtype(dtype) && H >= 1);
    const int64_t elt = dtype == MOE_BF16 ? 2 : 4;
    if ((H * elt) % 16 != 0) return MOE_ERR_UNSUPPORTED;
    row_vecs = H * elt / 16;
  }
  const size_t need = moe_permute_workspace(T, k, E);
  if (!workspace || ws_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255))
    return MOE_ERR_WORKSPACE;
  const int64_t nblk = ceil_div(P, kPermChunk);
  if (nblk > 0x7fffffff) return MOE_ERR_UNSUPPORTED;
  int32_t* counts = static_cast<int32_t*>(workspace);
  int32_t* bases = counts + nblk * E;
  hipStream_t st = as_stream(stream);
  PairSrc src{token_ids, topk_idx, n_tokens, k, E};
  perm_count_kernel<<<dim3((unsigned)nblk), dim3(kPermThreads), 0, st>>>(src, P, counts);
  MOE_CHECK_LAUNCH();
  perm_scan_kernel<<<dim3(1), dim3(256), 0, st>>>(counts, nblk, E, bases, expert_offsets);
  MOE_CHECK_LAUNCH();
  perm_rank_kernel<<<dim3((unsigned)nblk), dim3(kPermThreads), 0, st>>>(src, P, bases,
                                                                        row_of_pair, pair_of_row);
  MOE_CHECK_LAUNCH();
  if (x) {
    const int64_t gblocks = ceil_div(T, 4);
    if (gblocks > 0x7fffffff) return MOE_ERR_UNSUPPORTED;
    perm_gather_kernel<<<dim3((unsigned)gblocks), dim3(256), 0, st>>>(
        static_cast<const uint4*>(x), token_ids, T, n_tokens, k, row_vecs, row_of_pair, P,
        static_cast<uint4*>(x_perm));
    MOE_CHECK_LAUNCH();
  }
  return MOE_OK;
}
