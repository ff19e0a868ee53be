// moe_permute: stable expert-major grouping of (token, choice) pairs and the
// gather of hidden-state rows into that order.
//
// Three launches, all on the caller's stream, over chunks of ct consecutive
// batch tokens (ct * k pairs):
//   1. count          -- one block per chunk counts the experts of its pairs in
//                        an LDS histogram;
//   2. column scan    -- one block per expert turns that expert's counts over
//                        the chunks into each chunk's first row within the
//                        expert (exclusive scan) and the expert's total;
//   3. rank + gather  -- one block per chunk scans the expert totals into
//                        expert offsets, ranks its pairs stably (inside a
//                        wavefront, lanes holding the same expert are found with
//                        eight ballots, one per bit of the id, so a pair's rank
//                        is a popcount of the lower lanes in its match mask; wave
//                        totals carry across the block through LDS), writes both
//                        maps, then copies each of its tokens' rows once from x
//                        to its k destination rows with 16-byte vectors.
// ct is chosen on the host so that there are a few chunks per compute unit.
#include "common.h"

#include <algorithm>
#include <mutex>

namespace moe {
namespace {

constexpr int kPermThreads = 256;
constexpr int kMaxChunkPairs = 1024;   // pairs of one chunk, ranked in LDS
constexpr int64_t kSumInBlockCounts = 8192;   // (chunk, expert) counts a block sums itself

struct PairSrc {
  const int32_t* token_ids;
  const int32_t* idx;
  int64_t n_tokens;
  int k;
  int E;
};

// Token id of batch position i, or -1 when it is out of range.
__device__ __forceinline__ int64_t batch_token(const PairSrc& s, int64_t i) {
  const int64_t t = s.token_ids ? (int64_t)s.token_ids[i] : i;
  return (t >= 0 && t < s.n_tokens) ? t : -1;
}

// Expert of pair p, or -1 when the pair's token or expert id is out of range.
__device__ __forceinline__ int pair_expert(const PairSrc& s, int64_t p) {
  const int64_t i = p / s.k;
  const int j = (int)(p - i * s.k);
  const int64_t t = batch_token(s, i);
  if (t < 0) return -1;
  const int e = s.idx[t * s.k + j];
  return (e >= 0 && e < s.E) ? e : -1;
}

__device__ __forceinline__ int64_t ceil_div_dev(int64_t a, int64_t b) { return (a + b - 1) / b; }

template <int NT>
__device__ int block_excl_scan(int v, int* total) {
  __shared__ int s[NT / kWave];
  const int lane = lane_id();
  int x = v;
  for (int o = 1; o < kWave; o <<= 1) {
    const int y = __shfl_up(x, o, kWave);
    if (lane >= o) x += y;
  }
  if (lane == kWave - 1) s[threadIdx.x / kWave] = x;
  __syncthreads();
  int base = 0, tot = 0;
  for (int w = 0; w < NT / kWave; ++w) {
    if (w < (int)(threadIdx.x / kWave)) base += s[w];
    tot += s[w];
  }
  __syncthreads();
  *total = tot;
  return base + x - v;
}

__global__ void __launch_bounds__(kPermThreads)
perm_count_kernel(PairSrc src, int64_t P, int64_t chunk_pairs, int32_t* __restrict__ counts) {
  __shared__ int32_t hist[256];
  for (int e = threadIdx.x; e < src.E; e += blockDim.x) hist[e] = 0;
  __syncthreads();
  const int64_t start = (int64_t)blockIdx.x * chunk_pairs;
  const int64_t end = min(start + chunk_pairs, P);
  for (int64_t p = start + threadIdx.x; p < end; p += blockDim.x) {
    const int e = pair_expert(src, p);
    if (e >= 0) atomicAdd(&hist[e], 1);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < src.E; e += blockDim.x)
    counts[(int64_t)blockIdx.x * src.E + e] = hist[e];
}

// Per expert (one block each): first row within the expert of every chunk
// (exclusive scan of counts[:, e] over chunks) and the expert's total.
__global__ void __launch_bounds__(kPermThreads)
perm_colscan_kernel(const int32_t* __restrict__ counts, int64_t nchunks, int E,
                    int32_t* __restrict__ chunk_base, int32_t* __restrict__ totals) {
  const int e = blockIdx.x;
  const int64_t per = ceil_div_dev(nchunks, kPermThreads);
  const int64_t c0 = min(nchunks, (int64_t)threadIdx.x * per), c1 = min(nchunks, c0 + per);
  int32_t mine = 0;
  for (int64_t c = c0; c < c1; ++c) mine += counts[c * E + e];
  int total;
  int32_t run = block_excl_scan<kPermThreads>(mine, &total);
  for (int64_t c = c0; c < c1; ++c) {
    chunk_base[c * E + e] = run;
    run += counts[c * E + e];
  }
  if (threadIdx.x == 0) totals[e] = total;
}

// Workgroup barrier over LDS only: waits for this wave's LDS operations, not
// for its global loads, so row reads issued earlier stay in flight. The
// memory clobber keeps the compiler from moving loads or stores across it.
__device__ __forceinline__ void lds_sync() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int NT>
__device__ int block_excl_scan_lds(int v, int* total) {
  __shared__ int s[NT / kWave];
  const int lane = lane_id();
  int x = v;
  for (int o = 1; o < kWave; o <<= 1) {
    const int y = __shfl_up(x, o, kWave);
    if (lane >= o) x += y;
  }
  if (lane == kWave - 1) s[threadIdx.x / kWave] = x;
  lds_sync();
  int base = 0, tot = 0;
  for (int w = 0; w < NT / kWave; ++w) {
    if (w < (int)(threadIdx.x / kWave)) base += s[w];
    tot += s[w];
  }
  lds_sync();
  *total = tot;
  return base + x - v;
}

// Rows are moved as 16-byte vectors; row_vecs = row bytes / 16 (0: maps only).
// SUM_COUNTS: the block sums the per-chunk counts itself (few chunks x
// experts); otherwise chunk_base/totals come from perm_colscan_kernel.
// Global loads are issued in dependency order -- counts, the experts of the
// first 256 pairs, then the chunk's first rows of x -- and the ranking
// synchronises through LDS only, so the row reads overlap all index work.
template <bool SUM_COUNTS>
__global__ void __launch_bounds__(kPermThreads)
perm_rank_gather_kernel(PairSrc src, int64_t T, int64_t ct, int64_t nchunks,
                        const int32_t* __restrict__ counts, const int32_t* __restrict__ chunk_base,
                        const int32_t* __restrict__ totals, int32_t* __restrict__ expert_offsets,
                        int32_t* __restrict__ row_of_pair, int32_t* __restrict__ pair_of_row,
                        const uint4* __restrict__ x, int64_t row_vecs, uint4* __restrict__ x_perm) {
  constexpr int kWaves = kPermThreads / kWave;
  constexpr int kPrefetch = 16;                  // row vectors per thread loaded up front
  __shared__ int32_t tot[256], base[256];
  __shared__ int32_t wave_cnt[kWaves][256];
  __shared__ int32_t rows[kMaxChunkPairs];
  __shared__ int64_t tok[kMaxChunkPairs];
  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  const int E = src.E, k = src.k;
  const int64_t c = blockIdx.x;
  const int64_t i0 = c * ct, i1 = min(i0 + ct, T);
  const int64_t p0 = i0 * k, p1 = i1 * k;

  // 1. Index loads: count partials (thread tid sums expert tid % E over
  //    chunks g, g + G, ...; g = tid / E, G = 256 / E) or the scanned bases,
  //    the experts of the first round of pairs, and the chunk's token ids
  //    (into LDS, so the row loads below do not wait on them one by one).
  int32_t all = 0, bef = 0;
  const int G = kPermThreads / E;
  const int g = tid / E, ge = tid - g * E;
  if (SUM_COUNTS) {
    if (g < G) {
      // eight loads in flight per round
      int64_t cq = g;
      for (; cq + 7 * G < nchunks; cq += 8 * G) {
        int32_t v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = counts[(cq + u * G) * E + ge];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          all += v[u];
          bef += cq + u * G < c ? v[u] : 0;
        }
      }
      for (; cq < nchunks; cq += G) {
        const int32_t v = counts[cq * E + ge];
        all += v;
        bef += cq < c ? v : 0;
      }
    }
  } else if (tid < E) {
    all = totals[tid];
    bef = chunk_base[c * E + tid];
  }
  const int e_first = (p0 + tid < p1) ? pair_expert(src, p0 + tid) : -1;
  const int64_t ntok = i1 - i0;
  for (int64_t u = tid; u < ntok; u += kPermThreads) tok[u] = batch_token(src, i0 + u);
  lds_sync();

  // 2. The chunk's rows, flattened as f = u * row_vecs + v (token u, vector
  //    v): slot s of thread tid holds f = s * 256 + tid.
  // Slot positions (token u, vector v) advance by 256 flat positions per
  // slot; the token ids are read from LDS for all slots before any row load.
  const int64_t nf = ntok * row_vecs;
  const int64_t rv = row_vecs > 0 ? row_vecs : 1;
  const int64_t du = kPermThreads / rv, dv = kPermThreads - du * rv;
  int64_t su[kPrefetch], sv[kPrefetch];
  {
    int64_t u = tid / rv, v = tid - (tid / rv) * rv;
#pragma unroll
    for (int sl = 0; sl < kPrefetch; ++sl) {
      su[sl] = u;
      sv[sl] = v;
      u += du;
      v += dv;
      if (v >= rv) {
        v -= rv;
        ++u;
      }
    }
  }
  int64_t tv[kPrefetch];
#pragma unroll
  for (int sl = 0; sl < kPrefetch; ++sl) tv[sl] = tok[su[sl] < ntok ? su[sl] : 0];
  uint4 pf[kPrefetch];
#pragma unroll
  for (int sl = 0; sl < kPrefetch; ++sl) {
    const bool ok = row_vecs > 0 && su[sl] < ntok && tv[sl] >= 0;
    pf[sl] = ok ? x[tv[sl] * row_vecs + sv[sl]] : make_uint4(0, 0, 0, 0);
  }

  // 3. Expert offsets and this chunk's first row per expert.
  for (int e = tid; e < 256; e += kPermThreads) {
    tot[e] = 0;
    base[e] = 0;
    for (int w = 0; w < kWaves; ++w) wave_cnt[w][e] = 0;
  }
  lds_sync();
  if (SUM_COUNTS) {
    if (g < G) {
      atomicAdd(&tot[ge], all);
      atomicAdd(&base[ge], bef);
    }
  } else if (tid < E) {
    tot[tid] = all;
    base[tid] = bef;
  }
  lds_sync();
  int total;
  const int off = block_excl_scan_lds<kPermThreads>(tid < E ? tot[tid] : 0, &total);
  if (tid < E) {
    base[tid] += off;
    if (c == 0) expert_offsets[tid] = off;
  }
  if (c == 0 && tid == 0) expert_offsets[E] = total;
  lds_sync();

  // 4. Stable ranks of this chunk's pairs; base[] advances by each round.
  for (int64_t r0 = p0; r0 < p1; r0 += kPermThreads) {
    const int64_t p = r0 + tid;
    const int e = r0 == p0 ? e_first : ((p < p1) ? pair_expert(src, p) : -1);
    const bool valid = e >= 0;
    uint64_t match = ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const bool b = valid && ((e >> bit) & 1);
      const uint64_t bal = ballot(b);
      match &= b ? bal : ~bal;
    }
    const int rank_in_wave = __popcll(match & lanemask_lt());
    if (valid && (match & lanemask_lt()) == 0) wave_cnt[wave][e] = __popcll(match);
    lds_sync();
    if (p < p1) {
      int32_t row = -1;
      if (valid) {
        int32_t b = base[e];
        for (int w = 0; w < wave; ++w) b += wave_cnt[w][e];
        row = b + rank_in_wave;
        pair_of_row[row] = (int32_t)p;
      }
      row_of_pair[p] = row;
      rows[p - p0] = row;
    }
    lds_sync();
    for (int q = tid; q < E; q += kPermThreads) {
      int32_t add = 0;
      for (int w = 0; w < kWaves; ++w) {
        add += wave_cnt[w][q];
        wave_cnt[w][q] = 0;
      }
      base[q] += add;
    }
    lds_sync();
  }
  if (row_vecs == 0) return;

  // 5. Gather: each token row of the chunk is read once and written k times.
  auto put = [&](int64_t u, int64_t v, const uint4& val) {
    const int32_t* rr = rows + u * k;
    for (int j = 0; j < k; ++j) {
      const int32_t r = rr[j];
      if (r >= 0) x_perm[(int64_t)r * row_vecs + v] = val;
    }
  };
#pragma unroll
  for (int sl = 0; sl < kPrefetch; ++sl)
    if (su[sl] < ntok && tv[sl] >= 0) put(su[sl], sv[sl], pf[sl]);
  for (int64_t f = (int64_t)kPrefetch * kPermThreads + tid; f < nf; f += kPermThreads) {
    const int64_t u = f / row_vecs, v = f - u * row_vecs;
    const int64_t t = tok[u];
    if (t >= 0) put(u, v, x[t * row_vecs + v]);
  }
}

// Tokens per chunk: a power of two giving about two chunks per compute unit
// (512 chunks), at most kMaxChunkPairs pairs.
int64_t perm_chunk_tokens(int64_t T, int k) {
  const int64_t cap = std::max<int64_t>(1, kMaxChunkPairs / k);
  int64_t ct = 1;
  while (ct < cap && ct * 512 < T) ct *= 2;
  return ct;
}

}  // namespace
}  // namespace moe

extern "C" size_t moe_permute_workspace(int64_t T, int32_t k, int32_t E) {
  using namespace moe;
  if (T < 1 || k < 1 || E < 1) return 0;
  const int64_t nchunks = ceil_div(T, perm_chunk_tokens(T, k));
  return align_up((size_t)(2 * nchunks * E + E) * sizeof(int32_t), 256);
}

namespace moe {
namespace {

// Validation and launches shared by moe_permute and moe_permute_noalloc;
// `workspace` holds at least moe_permute_workspace(T, k, E) bytes.
int permute_run(const void* x, int32_t dtype, int64_t H, int64_t n_tokens,
                const int32_t* token_ids, int64_t T, const int32_t* topk_idx, int32_t k,
                int32_t E, int32_t* expert_offsets, int32_t* row_of_pair, int32_t* pair_of_row,
                void* x_perm, void* workspace, hipStream_t st) {
  const int64_t P = T * (int64_t)k;
  int64_t row_vecs = 0;
  if (x) row_vecs = H * (dtype == MOE_BF16 ? 2 : 4) / 16;
  const int64_t ct = perm_chunk_tokens(T, k);
  const int64_t nchunks = ceil_div(T, ct);
  if (nchunks > 0x7fffffff) return MOE_ERR_UNSUPPORTED;
  int32_t* counts = static_cast<int32_t*>(workspace);
  int32_t* chunk_base = counts + nchunks * E;
  int32_t* totals = chunk_base + nchunks * E;
  PairSrc src{token_ids, topk_idx, n_tokens, k, E};
  perm_count_kernel<<<dim3((unsigned)nchunks), dim3(kPermThreads), 0, st>>>(src, P, ct * k, counts);
  MOE_CHECK_LAUNCH();
  // Few (chunk, expert) counts: every block sums them itself; otherwise one
  // more launch scans them per expert.
  const bool sum_in_block = nchunks * E <= kSumInBlockCounts;
  if (sum_in_block) {
    perm_rank_gather_kernel<true><<<dim3((unsigned)nchunks), dim3(kPermThreads), 0, st>>>(
        src, T, ct, nchunks, counts, nullptr, nullptr, expert_offsets, row_of_pair, pair_of_row,
        static_cast<const uint4*>(x), row_vecs, static_cast<uint4*>(x_perm));
  } else {
    perm_colscan_kernel<<<dim3((unsigned)E), dim3(kPermThreads), 0, st>>>(counts, nchunks, E,
                                                                         chunk_base, totals);
    MOE_CHECK_LAUNCH();
    perm_rank_gather_kernel<false><<<dim3((unsigned)nchunks), dim3(kPermThreads), 0, st>>>(
        src, T, ct, nchunks, counts, chunk_base, totals, expert_offsets, row_of_pair,
        pair_of_row, static_cast<const uint4*>(x), row_vecs, static_cast<uint4*>(x_perm));
  }
  MOE_CHECK_LAUNCH();
  return MOE_OK;
}

// Host-side argument checks of both entry points (nothing is enqueued when
// they fail).
int permute_check(const void* x, int32_t dtype, int64_t H, int64_t n_tokens,
                  const int32_t* token_ids, int64_t T, const int32_t* topk_idx, int32_t k,
                  int32_t E, const int32_t* expert_offsets, const int32_t* row_of_pair,
                  const int32_t* pair_of_row, const void* x_perm) {
  MOE_CHECK_ARG(T >= 1 && k >= 1 && E >= 1 && E <= 256 && k <= E);
  MOE_CHECK_ARG(n_tokens >= 1 && (token_ids != nullptr || n_tokens >= T));
  MOE_CHECK_ARG(topk_idx && expert_offsets && row_of_pair && pair_of_row);
  MOE_CHECK_ARG((x == nullptr) == (x_perm == nullptr));
  MOE_CHECK_ARG(T * (int64_t)k < ((int64_t)1 << 31));
  if (x) {
    MOE_CHECK_ARG(valid_dtype(dtype) && H >= 1);
    const int64_t elt = dtype == MOE_BF16 ? 2 : 4;
    if ((H * elt) % 16 != 0) return MOE_ERR_UNSUPPORTED;
  }
  return MOE_OK;
}

}  // namespace
}  // namespace moe

extern "C" int moe_permute(const void* x, int32_t dtype, int64_t H, int64_t n_tokens,
                           const int32_t* token_ids, int64_t T, const int32_t* topk_idx,
                           int32_t k, int32_t E, int32_t* expert_offsets,
                           int32_t* row_of_pair, int32_t* pair_of_row, void* x_perm,
                           void* workspace, size_t ws_bytes, void* stream) {
  using namespace moe;
  const int rc = permute_check(x, dtype, H, n_tokens, token_ids, T, topk_idx, k, E,
                               expert_offsets, row_of_pair, pair_of_row, x_perm);
  if (rc != MOE_OK) return rc;
  const size_t need = moe_permute_workspace(T, k, E);
  if (!workspace || ws_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255))
    return MOE_ERR_WORKSPACE;
  return permute_run(x, dtype, H, n_tokens, token_ids, T, topk_idx, k, E, expert_offsets,
                     row_of_pair, pair_of_row, x_perm, workspace, as_stream(stream));
}

// ------------------------------------------------------------ no allocation
// moe_permute_noalloc takes its scratch from this array instead of a caller's
// workspace. Each device holds its own copy for the life of the process; host
// code never passes the array's name to a kernel (on the host it is only a
// stand-in for the symbol), only the device address looked up for the current
// device with hipGetSymbolAddress.
static __device__ __align__(256) int32_t scratch[MOE_PERMUTE_NOALLOC_SCRATCH_BYTES / 4];

namespace moe {
namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices];

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept.
hipError_t scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}
}  // namespace
}  // namespace moe

extern "C" int moe_permute_noalloc(const void* x, int32_t dtype, int64_t H, int64_t n_tokens,
                                   const int32_t* token_ids, int64_t T,
                                   const int32_t* topk_idx, int32_t k, int32_t E,
                                   int32_t* expert_offsets, int32_t* row_of_pair,
                                   int32_t* pair_of_row, void* x_perm, void* stream) {
  using namespace moe;
  const int rc = permute_check(x, dtype, H, n_tokens, token_ids, T, topk_idx, k, E,
                               expert_offsets, row_of_pair, pair_of_row, x_perm);
  if (rc != MOE_OK) return rc;
  if (moe_permute_workspace(T, k, E) > (size_t)MOE_PERMUTE_NOALLOC_SCRATCH_BYTES)
    return MOE_ERR_WORKSPACE;
  void* ws = nullptr;
  if (scratch_address(&ws) != hipSuccess) {
    (void)hipGetLastError();
    return MOE_ERR_HIP;
  }
  return permute_run(x, dtype, H, n_tokens, token_ids, T, topk_idx, k, E, expert_offsets,
                     row_of_pair, pair_of_row, x_perm, ws, as_stream(stream));
}
