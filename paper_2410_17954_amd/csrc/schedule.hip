// moe_schedule: the Token Scheduler of Sec. 3.3 -- balanced rebatching of two
// adjacent batches by predicted routing path, approximating Eq. 2 with the
// two-centroid clustering of Sec. 3.3.2 under S_ij = 1 - d_ij / (L E).
//
// S_ij falls as the Hamming distance d_ij grows, so every step is integer:
//   pack     routes -> packed paths, bit l*E+e of token i set iff expert e is
//            among its choices at layer l (W = ceil(L E / 64) words per token)
//   order    signature order: ascending per-layer expert ids, layer 0 first,
//            then token index. For two paths with the same number of ids per
//            layer, a precedes b iff the lowest bit where they differ is set in
//            a, so the order is decided word by word on the packed paths. The
//            rank of each token is counted in parallel over (i, j-tile) pairs.
//   init     m1 = argmin_i sum_j d_ij over all tokens, m2 = argmax_i d(i, m1)
//   iterate  delta_i = d(i,m1) - d(i,m2) and its histogram; the threshold
//            delta* where the count reaches n1; batch 1 = delta < delta* plus
//            the first tokens at delta* in signature order; per-batch column
//            counts c_b; sum_{j in C} d_ij = |C| |r_i| + sum_j |r_j|
//            - 2 sum_{b in r_i} c_b; per-batch argmin -> new centroids;
//            a device-side flag stops the remaining rounds once they settle
//   finish   Eq. 2 before/after from the column counts, the optional guard,
//            perm by stable compaction, demand, info.
// All ties go to the lower signature rank. The launch sequence is fixed
// (12 + 5 * max_iters launches); nothing is read back to the host.
#include "common.h"

#include <algorithm>

namespace moe {
namespace {

constexpr int kT = 256;          // threads of grid-parallel kernels
constexpr int kSel = 1024;       // threads of single-block kernels
constexpr int kRankTile = 1024;  // j-tile of the rank count

// state words
enum {
  ST_M1 = 0, ST_M2, ST_DONE, ST_ITERS, ST_CONV, ST_AM1, ST_AM2, ST_TOT0, ST_TOT1, ST_NWORDS = 16
};

struct Cand {
  int64_t v;
  int32_t rank;
  int32_t idx;
};

__device__ __forceinline__ bool cand_less(const Cand& a, const Cand& b) {
  return a.v < b.v || (a.v == b.v && a.rank < b.rank);
}

__device__ __forceinline__ Cand cand_none() { return Cand{INT64_MAX, INT32_MAX, -1}; }

__device__ __forceinline__ Cand wave_min(Cand c) {
  for (int o = 32; o > 0; o >>= 1) {
    Cand d;
    d.v = __shfl_xor(c.v, o, kWave);
    d.rank = __shfl_xor(c.rank, o, kWave);
    d.idx = __shfl_xor(c.idx, o, kWave);
    if (cand_less(d, c)) c = d;
  }
  return c;
}

// Block-wide min of candidates; result valid in every thread.
template <int NT>
__device__ Cand block_min(Cand c) {
  __shared__ Cand s[NT / kWave];
  c = wave_min(c);
  if (lane_id() == 0) s[threadIdx.x / kWave] = c;
  __syncthreads();
  Cand r = s[0];
  for (int w = 1; w < NT / kWave; ++w)
    if (cand_less(s[w], r)) r = s[w];
  __syncthreads();
  return r;
}

// Exclusive scan of one int per thread across a block of NT threads; also
// returns the block total.
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

__device__ __forceinline__ uint64_t lowbit(uint64_t d) { return d & (0ull - d); }

// ---------------------------------------------------------------- kernels
__global__ void __launch_bounds__(kT)
sch_pack(const uint8_t* __restrict__ routes, int N, int L, int E, int k, int W,
         uint64_t* __restrict__ bits, uint64_t* __restrict__ bits_t, int32_t* __restrict__ ones,
         int32_t* __restrict__ rank) {
  const int i = blockIdx.x * kT + threadIdx.x;
  if (i >= N) return;
  rank[i] = 0;
  uint64_t* b = bits + (int64_t)i * W;
  for (int w = 0; w < W; ++w) b[w] = 0;
  const uint8_t* r = routes + (int64_t)i * L * k;
  for (int l = 0; l < L; ++l)
    for (int j = 0; j < k; ++j) {
      const int e = r[l * k + j];
      if (e < E) {
        const int64_t bit = (int64_t)l * E + e;
        b[bit >> 6] |= 1ull << (bit & 63);
      }
    }
  int c = 0;
  for (int w = 0; w < W; ++w) {
    c += __popcll(b[w]);
    bits_t[(int64_t)w * N + i] = b[w];          // word-major copy: coalesced per word
  }
  ones[i] = c;
}

// rank[i] += #{j in this tile : j precedes i in signature order}
__global__ void __launch_bounds__(kT)
sch_rank(const uint64_t* __restrict__ bits, int N, int W, int32_t* __restrict__ rank) {
  __shared__ uint64_t s_w0[kRankTile];
  const int j0 = blockIdx.y * kRankTile;
  const int jn = min(kRankTile, N - j0);
  for (int q = threadIdx.x; q < jn; q += kT) s_w0[q] = bits[(int64_t)(j0 + q) * W];
  __syncthreads();
  const int i = blockIdx.x * kT + threadIdx.x;
  if (i >= N) return;
  const uint64_t wi = bits[(int64_t)i * W];
  int cnt = 0;
  for (int q = 0; q < jn; ++q) {
    const uint64_t wj = s_w0[q];
    const uint64_t d = wi ^ wj;
    if (d) {
      cnt += (wj & lowbit(d)) != 0;
    } else {
      const int j = j0 + q;
      if (j == i) continue;
      int before = j < i;
      for (int w = 1; w < W; ++w) {
        const uint64_t a = bits[(int64_t)j * W + w];
        const uint64_t dd = a ^ bits[(int64_t)i * W + w];
        if (dd) {
          before = (a & lowbit(dd)) != 0;
          break;
        }
      }
      cnt += before;
    }
  }
  atomicAdd(&rank[i], cnt);
}

__global__ void __launch_bounds__(kT)
sch_order(const int32_t* __restrict__ rank, int N, int32_t* __restrict__ order) {
  const int i = blockIdx.x * kT + threadIdx.x;
  if (i < N) order[rank[i]] = i;
}

// Column counts. mode 0: all tokens -> cnt[0]; mode 1: original split
// (i < n1 -> cnt[0], else cnt[1]); mode 2: current batches (in1[i] -> cnt[0]).
// tot[c] accumulates |r_i| of the tokens counted into cnt[c].
__global__ void __launch_bounds__(kT)
sch_colcount(const uint64_t* __restrict__ bits, const int32_t* __restrict__ ones, int N, int W,
             int LE, int mode, int n1, const int32_t* __restrict__ in1,
             int32_t* __restrict__ cnt, unsigned long long* __restrict__ tot,
             const int64_t* __restrict__ state) {
  extern __shared__ int32_t s_cnt[];           // 2 * LE when it fits, else unused
  if (mode == 2 && state[ST_DONE]) return;
  const bool priv = (2 * LE) <= 8192;
  if (priv) {
    for (int b = threadIdx.x; b < 2 * LE; b += kT) s_cnt[b] = 0;
    __syncthreads();
  }
  const int i = blockIdx.x * kT + threadIdx.x;
  int c = 0;
  if (i < N) {
    c = mode == 0 ? 0 : (mode == 1 ? (i < n1 ? 0 : 1) : (in1[i] ? 0 : 1));
    int32_t* dst = priv ? s_cnt + c * LE : cnt + c * LE;
    for (int w = 0; w < W; ++w) {
      uint64_t word = bits[(int64_t)i * W + w];
      while (word) {
        const int b = w * 64 + __builtin_ctzll(word);
        atomicAdd(&dst[b], 1);
        word &= word - 1;
      }
    }
  }
  // per-block |r_i| sums for each batch
  int o0 = (i < N && c == 0) ? ones[i] : 0;
  int o1 = (i < N && c == 1) ? ones[i] : 0;
  o0 = wave_sum(o0);
  o1 = wave_sum(o1);
  if (lane_id() == 0) {
    if (o0) atomicAdd(&tot[0], (unsigned long long)o0);
    if (o1) atomicAdd(&tot[1], (unsigned long long)o1);
  }
  if (priv) {
    __syncthreads();
    for (int b = threadIdx.x; b < 2 * LE; b += kT)
      if (s_cnt[b]) atomicAdd(&cnt[b], s_cnt[b]);
  }
}

// Per-block argmin candidates. mode 0: total distance to all tokens (one
// batch of N); mode 1: farthest from m1 (value = -d(i, m1), i != m1);
// mode 2: total distance to the members of the token's own batch.
__global__ void __launch_bounds__(kT)
sch_cand(const uint64_t* __restrict__ bits, const int32_t* __restrict__ ones,
         const int32_t* __restrict__ rank, int N, int W, int LE, int mode, int n1,
         const int32_t* __restrict__ in1, const int32_t* __restrict__ cnt,
         const unsigned long long* __restrict__ tot, const int64_t* __restrict__ state,
         Cand* __restrict__ cand) {
  if (mode == 2 && state[ST_DONE]) return;
  const int i = blockIdx.x * kT + threadIdx.x;
  Cand c0 = cand_none(), c1 = cand_none();
  if (i < N) {
    const uint64_t* bi = bits + (int64_t)i * W;
    if (mode == 1) {
      const int m1 = (int)state[ST_M1];
      if (i != m1) {
        const uint64_t* bm = bits + (int64_t)m1 * W;
        int d = 0;
        for (int w = 0; w < W; ++w) d += __popcll(bi[w] ^ bm[w]);
        c0 = Cand{-(int64_t)d, rank[i], i};
      }
    } else {
      const int c = mode == 0 ? 0 : (in1[i] ? 0 : 1);
      const int64_t size = mode == 0 ? N : (c == 0 ? n1 : N - n1);
      const int32_t* cc = cnt + c * LE;
      int64_t g = 0;
      for (int w = 0; w < W; ++w) {
        uint64_t word = bi[w];
        while (word) {
          g += cc[w * 64 + __builtin_ctzll(word)];
          word &= word - 1;
        }
      }
      const int64_t D = size * ones[i] + (int64_t)tot[c] - 2 * g;
      const Cand me{D, rank[i], i};
      if (c == 0) c0 = me; else c1 = me;
    }
  }
  const Cand r0 = block_min<kT>(c0);
  const Cand r1 = block_min<kT>(c1);
  if (threadIdx.x == 0) {
    cand[2 * blockIdx.x] = r0;
    cand[2 * blockIdx.x + 1] = r1;
  }
}

// Reduce the per-block candidates. mode 0: set m1; mode 1: set m2;
// mode 2: centroid update + convergence test.
__global__ void __launch_bounds__(kSel)
sch_pick(const Cand* __restrict__ cand, int nblk, int mode, int64_t* __restrict__ state) {
  if (mode == 2 && state[ST_DONE]) return;
  Cand c0 = cand_none(), c1 = cand_none();
  for (int b = threadIdx.x; b < nblk; b += kSel) {
    if (cand_less(cand[2 * b], c0)) c0 = cand[2 * b];
    if (cand_less(cand[2 * b + 1], c1)) c1 = cand[2 * b + 1];
  }
  c0 = block_min<kSel>(c0);
  c1 = block_min<kSel>(c1);
  if (threadIdx.x != 0) return;
  if (mode == 0) {
    state[ST_M1] = c0.idx;
  } else if (mode == 1) {
    state[ST_M2] = c0.idx;
  } else {
    state[ST_ITERS] += 1;
    if (c0.idx == state[ST_M1] && c1.idx == state[ST_M2]) {
      state[ST_CONV] = 1;
      state[ST_DONE] = 1;
    } else {
      state[ST_M1] = c0.idx;
      state[ST_M2] = c1.idx;
    }
  }
}

__global__ void __launch_bounds__(kT)
sch_delta(const uint64_t* __restrict__ bits, int N, int W, int off,
          int32_t* __restrict__ delta, int32_t* __restrict__ hist,
          const int64_t* __restrict__ state) {
  if (state[ST_DONE]) return;
  const int i = blockIdx.x * kT + threadIdx.x;
  if (i >= N) return;
  const uint64_t* bi = bits + (int64_t)i * W;
  const uint64_t* b1 = bits + state[ST_M1] * W;
  const uint64_t* b2 = bits + state[ST_M2] * W;
  int d = 0;
  for (int w = 0; w < W; ++w) d += __popcll(bi[w] ^ b1[w]) - __popcll(bi[w] ^ b2[w]);
  delta[i] = d;
  atomicAdd(&hist[d + off], 1);
}

// Balanced assignment: the n1 smallest (delta, signature rank) go to batch 1.
// Also clears the histogram and the batch column counts for their next use.
__global__ void __launch_bounds__(kSel)
sch_select(int N, int n1, int nbins, int off, const int32_t* __restrict__ delta,
           const int32_t* __restrict__ order, int32_t* __restrict__ hist,
           int32_t* __restrict__ in1, int32_t* __restrict__ cnt, int LE,
           unsigned long long* __restrict__ tot, int64_t* __restrict__ state) {
  if (state[ST_DONE]) return;
  __shared__ int s_thr, s_q;
  if (threadIdx.x == 0) {
    int cum = 0, thr = nbins - 1 - off, q = n1;
    for (int v = 0; v < nbins; ++v) {
      const int h = hist[v];
      if (cum + h >= n1) {
        thr = v - off;
        q = n1 - cum;
        break;
      }
      cum += h;
    }
    s_thr = thr;
    s_q = q;
    state[ST_AM1] = state[ST_M1];
    state[ST_AM2] = state[ST_M2];
    tot[0] = 0;
    tot[1] = 0;
  }
  __syncthreads();
  for (int v = threadIdx.x; v < nbins; v += kSel) hist[v] = 0;
  for (int b = threadIdx.x; b < 2 * LE; b += kSel) cnt[b] = 0;
  const int thr = s_thr, q = s_q;
  const int per = (N + kSel - 1) / kSel;
  const int r0 = min(N, (int)threadIdx.x * per), r1 = min(N, r0 + per);
  int ties = 0;
  for (int r = r0; r < r1; ++r) {
    const int i = order[r];
    ties += (i >= 0 && i < N) && delta[i] == thr;
  }
  int total;
  int pre = block_excl_scan<kSel>(ties, &total);
  for (int r = r0; r < r1; ++r) {
    const int i = order[r];
    if (i < 0 || i >= N) continue;
    const int d = delta[i];
    int v;
    if (d < thr) v = 1;
    else if (d > thr) v = 0;
    else v = (pre++ < q) ? 1 : 0;
    in1[i] = v;
  }
}

__global__ void __launch_bounds__(kSel)
sch_finish(int N, int n1, int L, int E, int keep_if_worse, int trivial,
           const int32_t* __restrict__ in1, const int32_t* __restrict__ cnt,
           const int32_t* __restrict__ cnt_orig, const int64_t* __restrict__ state,
           const int32_t* __restrict__ err,
           int32_t* __restrict__ perm, int32_t* __restrict__ demand, int64_t* __restrict__ info) {
  const int LE = L * E;
  int a = 0, b = 0;
  for (int q = threadIdx.x; q < LE; q += kSel) {
    a += (cnt_orig[q] > 0) + (cnt_orig[LE + q] > 0);
    if (!trivial) b += (cnt[q] > 0) + (cnt[LE + q] > 0);
  }
  int before, after;
  block_excl_scan<kSel>(a, &before);
  block_excl_scan<kSel>(b, &after);
  if (trivial) after = before;
  const bool use_orig = trivial || (keep_if_worse && after > before);
  const int32_t* src = use_orig ? cnt_orig : cnt;
  // stable compaction: batch 1 in ascending index, then batch 2
  const int per = (N + kSel - 1) / kSel;
  const int i0 = min(N, (int)threadIdx.x * per), i1 = min(N, i0 + per);
  int mine = 0;
  for (int i = i0; i < i1; ++i) mine += use_orig ? (i < n1) : (in1[i] != 0);
  int tot1;
  int p1 = block_excl_scan<kSel>(mine, &tot1);
  int p2 = tot1 + (i0 - p1);
  for (int i = i0; i < i1; ++i) {
    const bool one = use_orig ? (i < n1) : (in1[i] != 0);
    if (one) perm[p1++] = i;
    else perm[p2++] = i;
  }
  if (demand)
    for (int q = threadIdx.x; q < 2 * LE; q += kSel) demand[q] = src[q];
  if (threadIdx.x == 0) {
    // a bounded wait that timed out in the cooperative loop marks the result
    info[0] = (*err) ? -1 : (trivial ? 0 : state[ST_ITERS]);
    info[1] = trivial ? 1 : state[ST_CONV];
    info[2] = trivial ? -1 : state[ST_AM1];
    info[3] = trivial ? -1 : state[ST_AM2];
    info[4] = before;
    info[5] = use_orig ? before : after;
    info[6] = (!trivial && use_orig) ? 1 : 0;
    info[7] = n1;
  }
}

// ------------------------------------------------ rank with keys in LDS
// Same count as sch_rank, with the whole key of every token of the j-tile
// staged in LDS and token i's key in registers (W <= WMAX words), so equal
// leading words never go back to global memory.
template <int WMAX>
__global__ void __launch_bounds__(kT)
sch_rank_keys(const uint64_t* __restrict__ bits, int N, int W, int tile,
              int32_t* __restrict__ rank) {
  extern __shared__ uint64_t s_keys[];          // [tile][W]
  const int j0 = blockIdx.y * tile;
  const int jn = min(tile, N - j0);
  for (int q = threadIdx.x; q < jn * W; q += kT) s_keys[q] = bits[(int64_t)j0 * W + q];
  __syncthreads();
  const int i = blockIdx.x * kT + threadIdx.x;
  if (i >= N) return;
  uint64_t ki[WMAX];
#pragma unroll
  for (int w = 0; w < WMAX; ++w) ki[w] = (w < W) ? bits[(int64_t)i * W + w] : 0ull;
  // Most pairs differ in their first word; the remaining words are compared
  // only on a tie there (all still in LDS / registers).
  auto before = [&](int q) -> int {
    const uint64_t* kj = s_keys + q * W;
    const uint64_t a0 = kj[0];
    const uint64_t d0 = a0 ^ ki[0];
    if (d0) return (a0 & lowbit(d0)) != 0;
#pragma unroll
    for (int w = 1; w < WMAX; ++w) {
      if (w < W) {
        const uint64_t a = kj[w];
        const uint64_t d = a ^ ki[w];
        if (d) return (a & lowbit(d)) != 0;
      }
    }
    return (j0 + q) < i;                          // equal keys: index order; j == i adds 0
  };
  int cnt = 0;
  int q = 0;
  for (; q + 4 <= jn; q += 4) cnt += before(q) + before(q + 1) + before(q + 2) + before(q + 3);
  for (; q < jn; ++q) cnt += before(q);
  atomicAdd(&rank[i], cnt);
}

// ------------------------------------------------ cooperative round loop
// All rounds in one cooperative launch (every block resident): block b owns
// a contiguous range of token indices and the same range of signature ranks.
// Data that crosses blocks inside the launch is read and written with
// device-scope atomics, and phases are separated by a grid barrier on a
// monotonic arrival counter: every thread issues an agent-scope release fence
// before its block arrives (the XCD L2s are not coherent with each other, and
// a workgroup barrier does not wait for the other waves' memory operations)
// and an acquire fence after the wait. Every barrier wait is
// bounded: past the bound the block records an error and goes on, so the
// launch always terminates (the result is then flagged, never trusted).
// Candidates are packed as (value << 24 | signature rank) and reduced with a
// 64-bit atomicMin, which keeps the lower-rank tie rule.
constexpr int kCoopT = 256;
constexpr int kCoopMaxLE = 8192;
constexpr unsigned kSpinBound = 1u << 20;

// Shared data within the launch: reads as an atomic add of zero, writes as an
// atomic exchange, the same path the accumulating atomics take.
__device__ __forceinline__ int ld_coh(const int32_t* p) {
  return atomicAdd(const_cast<int32_t*>(p), 0);
}
__device__ __forceinline__ void st_coh(int32_t* p, int32_t v) { atomicExch(p, v); }
__device__ __forceinline__ unsigned long long ld_coh64(const unsigned long long* p) {
  return atomicAdd(const_cast<unsigned long long*>(p), 0ull);
}
__device__ __forceinline__ void st_coh64(unsigned long long* p, unsigned long long v) {
  atomicExch(p, v);
}

__device__ void grid_sync(unsigned* bar, unsigned nblk, int32_t* err) {
  // Release: every wave waits for its own stores and atomics and writes the
  // XCD's L2 back, so the arrival below is ordered after all of them (a
  // workgroup barrier alone does not wait for other waves' memory traffic).
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned arrived = atomicAdd(bar, 1u) + 1u;
    const unsigned target = (arrived + nblk - 1u) / nblk * nblk;
    unsigned spins = 0;
    while (atomicAdd(bar, 0u) < target) {
      __builtin_amdgcn_s_sleep(1);
      if (++spins == kSpinBound) {
        atomicExch(err, 1);
        break;
      }
    }
  }
  __syncthreads();
  __threadfence();                               // acquire: drop stale cached lines
}

__device__ __forceinline__ unsigned long long wave_min_u64(unsigned long long v) {
  for (int o = 32; o > 0; o >>= 1) {
    const unsigned long long w = __shfl_xor(v, o, kWave);
    v = w < v ? w : v;
  }
  return v;
}

struct CoopArgs {
  const uint64_t* bits_t;   // [W][N] word-major paths
  const int32_t* ones;
  const int32_t* rank;
  const int32_t* order;
  int N, W, LE, n1, nbins, off, max_iters, trivial, twoLk;
  int32_t* delta;           // [N]
  int32_t* in1;             // [N]
  int32_t* hist;            // [nbins]
  int32_t* cnt;             // [2][LE]
  int32_t* cnt_orig;        // [2][LE]
  unsigned long long* tot;  // [4]: batch sums, then input-split sums
  unsigned long long* cand; // [2]
  int32_t* tiecnt;          // [nblk]
  unsigned* bar;
  int32_t* err;
  int64_t* state;
};

__global__ void __launch_bounds__(kCoopT)
sch_coop(CoopArgs a) {
  __shared__ int32_t s_c[2 * kCoopMaxLE];        // local column counts / copy of cnt
  __shared__ uint64_t s_med[2][kCoopMaxLE / 64];
  __shared__ unsigned long long s_red[kCoopT / kWave];
  __shared__ int s_thr, s_q;
  __shared__ unsigned long long s_tot[2];
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const unsigned nblk = gridDim.x;
  const int N = a.N, W = a.W, LE = a.LE;
  const int per = (N + (int)nblk - 1) / (int)nblk;
  const int t0 = min(N, (int)blockIdx.x * per), t1 = min(N, t0 + per);

  auto word = [&](int i, int w) { return a.bits_t[(int64_t)w * N + i]; };

  auto block_min_u64 = [&](unsigned long long v) {
    v = wave_min_u64(v);
    if (lane == 0) s_red[tid / kWave] = v;
    __syncthreads();
    unsigned long long r = s_red[0];
    for (int w = 1; w < kCoopT / kWave; ++w) r = s_red[w] < r ? s_red[w] : r;
    __syncthreads();
    return r;
  };

  // Column counts of this block's tokens into global cnt (batch of token i
  // from `batch_of`), plus |r| sums into tot[2 * which + batch].
  auto count = [&](auto batch_of, int32_t* dst, int which) {
    for (int q = tid; q < 2 * LE; q += kCoopT) s_c[q] = 0;
    if (tid < 2) s_tot[tid] = 0;
    __syncthreads();
    for (int i = t0 + tid; i < t1; i += kCoopT) {
      const int c = batch_of(i);
      for (int w = 0; w < W; ++w) {
        uint64_t x = word(i, w);
        while (x) {
          atomicAdd(&s_c[c * LE + w * 64 + __builtin_ctzll(x)], 1);
          x &= x - 1;
        }
      }
      atomicAdd(&s_tot[c], (unsigned long long)a.ones[i]);
    }
    __syncthreads();
    for (int q = tid; q < 2 * LE; q += kCoopT)
      if (s_c[q]) atomicAdd(&dst[q], s_c[q]);
    if (tid < 2 && s_tot[tid]) atomicAdd(&a.tot[2 * which + tid], s_tot[tid]);
  };

  // Candidate key of token i under the batch sums copied into s_c / s_tot.
  auto dist_key = [&](int i, int c, int64_t size) -> unsigned long long {
    const int32_t* cc = s_c + c * LE;
    int64_t g = 0;
    for (int w = 0; w < W; ++w) {
      uint64_t x = word(i, w);
      while (x) {
        g += cc[w * 64 + __builtin_ctzll(x)];
        x &= x - 1;
      }
    }
    const int64_t D = size * a.ones[i] + (int64_t)s_tot[c] - 2 * g;
    return ((unsigned long long)D << 24) | (unsigned long long)a.rank[i];
  };

  // ---- input split: column counts (Eq. 2 before, demand of the original)
  count([&](int i) { return i < a.n1 ? 0 : 1; }, a.cnt_orig, 1);
  if (a.trivial) return;                          // uniform over the grid
  grid_sync(a.bar, nblk, a.err);

  // ---- m1: least total distance; counts over everyone = both input batches
  for (int q = tid; q < LE; q += kCoopT) s_c[q] = ld_coh(a.cnt_orig + q) + ld_coh(a.cnt_orig + LE + q);
  if (tid == 0) s_tot[0] = ld_coh64(a.tot + 2) + ld_coh64(a.tot + 3);
  __syncthreads();
  {
    unsigned long long best = ~0ull;
    for (int i = t0 + tid; i < t1; i += kCoopT) {
      const unsigned long long k = dist_key(i, 0, N);
      best = k < best ? k : best;
    }
    best = block_min_u64(best);
    if (tid == 0) atomicMin(&a.cand[0], best);
  }
  grid_sync(a.bar, nblk, a.err);
  auto decode = [&](unsigned long long key) {
    const int r = (int)(key & 0xFFFFFF);
    return r < N ? a.order[r] : 0;               // empty batch only after a barrier error
  };
  int m1 = decode(ld_coh64(a.cand));
  for (int w = tid; w < W; w += kCoopT) s_med[0][w] = word(m1, w);
  __syncthreads();
  // ---- m2: farthest from m1, as a minimum of (2Lk - d, rank)
  {
    unsigned long long best = ~0ull;
    for (int i = t0 + tid; i < t1; i += kCoopT) {
      if (i == m1) continue;
      int d = 0;
      for (int w = 0; w < W; ++w) d += __popcll(word(i, w) ^ s_med[0][w]);
      const unsigned long long k = ((unsigned long long)(a.twoLk - d) << 24) | (unsigned long long)a.rank[i];
      best = k < best ? k : best;
    }
    best = block_min_u64(best);
    if (tid == 0) atomicMin(&a.cand[1], best);
  }
  grid_sync(a.bar, nblk, a.err);
  int m2 = decode(ld_coh64(a.cand + 1));

  int iters = 0, conv = 0, am1 = -1, am2 = -1;
  for (int it = 1; it <= a.max_iters; ++it) {
    // A: delta_i = d(i, m1) - d(i, m2) for own tokens, histogram
    for (int w = tid; w < W; w += kCoopT) {
      s_med[0][w] = word(m1, w);
      s_med[1][w] = word(m2, w);
    }
    __syncthreads();
    for (int i = t0 + tid; i < t1; i += kCoopT) {
      int d = 0;
      for (int w = 0; w < W; ++w) {
        const uint64_t x = word(i, w);
        d += __popcll(x ^ s_med[0][w]) - __popcll(x ^ s_med[1][w]);
      }
      st_coh(a.delta + i, d);
      atomicAdd(&a.hist[d + a.off], 1);
    }
    grid_sync(a.bar, nblk, a.err);
    // B: threshold (every block alike), ties of own rank range; resets
    {
      const int pb = (a.nbins + kCoopT - 1) / kCoopT;
      const int v0 = min(a.nbins, tid * pb), v1 = min(a.nbins, v0 + pb);
      int local = 0;
      for (int v = v0; v < v1; ++v) local += ld_coh(a.hist + v);
      int total;
      int cum = block_excl_scan<kCoopT>(local, &total);
      for (int v = v0; v < v1; ++v) {
        const int h = ld_coh(a.hist + v);
        if (cum < a.n1 && cum + h >= a.n1) {
          s_thr = v - a.off;
          s_q = a.n1 - cum;
        }
        cum += h;
      }
    }
    __syncthreads();
    const int thr = s_thr, q = s_q;
    const int sub = (t1 - t0 + kCoopT - 1) / kCoopT;      // ranks per thread
    const int r0 = min(t1, t0 + tid * sub), r1 = min(t1, r0 + sub);
    int ties = 0;
    for (int r = r0; r < r1; ++r) ties += ld_coh(a.delta + a.order[r]) == thr;
    int btot;
    int pre_in_block = block_excl_scan<kCoopT>(ties, &btot);
    if (tid == 0) st_coh(a.tiecnt + blockIdx.x, btot);
    if (blockIdx.x == 0) {
      if (tid < 2) st_coh64(a.cand + tid, ~0ull);
      if (tid < 2) st_coh64(a.tot + tid, 0ull);
    }
    for (int qq = blockIdx.x * kCoopT + tid; qq < 2 * LE; qq += (int)nblk * kCoopT) st_coh(a.cnt + qq, 0);
    grid_sync(a.bar, nblk, a.err);
    // C: the first n1 in (delta, rank) order go to batch 1; hist reset
    {
      int before = 0;
      for (unsigned b = 0; b < blockIdx.x; ++b) before += ld_coh(a.tiecnt + b);
      int pre = before + pre_in_block;
      for (int r = r0; r < r1; ++r) {
        const int i = a.order[r];
        const int d = ld_coh(a.delta + i);
        st_coh(a.in1 + i, d < thr ? 1 : (d > thr ? 0 : (pre++ < q ? 1 : 0)));
      }
    }
    for (int v = blockIdx.x * kCoopT + tid; v < a.nbins; v += (int)nblk * kCoopT) st_coh(a.hist + v, 0);
    am1 = m1;
    am2 = m2;
    iters = it;
    grid_sync(a.bar, nblk, a.err);
    // D: batch column counts
    count([&](int i) { return ld_coh(a.in1 + i) ? 0 : 1; }, a.cnt, 0);
    grid_sync(a.bar, nblk, a.err);
    // E: centroid candidates per batch
    for (int qq = tid; qq < 2 * LE; qq += kCoopT) s_c[qq] = ld_coh(a.cnt + qq);
    if (tid < 2) s_tot[tid] = ld_coh64(a.tot + tid);
    __syncthreads();
    {
      unsigned long long b0 = ~0ull, b1 = ~0ull;
      for (int i = t0 + tid; i < t1; i += kCoopT) {
        const int c = ld_coh(a.in1 + i) ? 0 : 1;
        const unsigned long long k = dist_key(i, c, c == 0 ? a.n1 : N - a.n1);
        if (c == 0) b0 = k < b0 ? k : b0;
        else b1 = k < b1 ? k : b1;
      }
      b0 = block_min_u64(b0);
      b1 = block_min_u64(b1);
      if (tid == 0) {
        atomicMin(&a.cand[0], b0);
        atomicMin(&a.cand[1], b1);
      }
    }
    grid_sync(a.bar, nblk, a.err);
    // F: new centroids; stop when they repeat (same decision in every block)
    const int n1c = decode(ld_coh64(a.cand));
    const int n2c = decode(ld_coh64(a.cand + 1));
    if (n1c == m1 && n2c == m2) {
      conv = 1;
      break;
    }
    m1 = n1c;
    m2 = n2c;
  }
  if (blockIdx.x == 0 && tid == 0) {
    a.state[ST_ITERS] = iters;
    a.state[ST_CONV] = conv;
    a.state[ST_AM1] = am1;
    a.state[ST_AM2] = am2;
  }
}

// Clears the small scratch of one call (a kernel rather than memset nodes,
// so that the sequence can be captured in a graph).
__global__ void __launch_bounds__(kT)
sch_init(int32_t* __restrict__ hist, int nbins, int32_t* __restrict__ cnt_orig, int LE2,
         unsigned long long* __restrict__ tot, unsigned long long* __restrict__ cand,
         unsigned* __restrict__ bar, int32_t* __restrict__ err, int64_t* __restrict__ state) {
  const int g = blockIdx.x * kT + threadIdx.x, stride = gridDim.x * kT;
  for (int q = g; q < nbins; q += stride) hist[q] = 0;
  for (int q = g; q < LE2; q += stride) cnt_orig[q] = 0;
  if (g < 4) tot[g] = 0;
  if (g < 2) cand[g] = ~0ull;
  if (g < ST_NWORDS) state[g] = 0;
  if (g == 0) {
    *bar = 0;
    *err = 0;
  }
}

struct SchLayout {
  size_t bits, bits_t, ones, rank, order, delta, in1, cnt, cnt_orig, hist, tot, state, cand,
      cand2, tiecnt, bar, total;
};

SchLayout sch_layout(int64_t N, int32_t L, int32_t E, int32_t k) {
  const int64_t W = ((int64_t)L * E + 63) / 64;
  const int64_t LE = (int64_t)L * E;
  const int64_t nbins = 4 * (int64_t)L * k + 1;
  const int64_t nblk = ceil_div(N, kT);
  SchLayout s{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + bytes, 256);
    return at;
  };
  s.bits = take(N * W * 8);
  s.bits_t = take(N * W * 8);
  s.ones = take(N * 4);
  s.rank = take(N * 4);
  s.order = take(N * 4);
  s.delta = take(N * 4);
  s.in1 = take(N * 4);
  s.cnt = take(2 * LE * 4);
  s.cnt_orig = take(2 * LE * 4);
  s.hist = take(nbins * 4);
  s.tot = take(4 * 8);
  s.state = take(ST_NWORDS * 8);
  s.cand = take(nblk * 2 * sizeof(Cand));
  s.cand2 = take(2 * 8);
  s.tiecnt = take(nblk * 4);
  s.bar = take(2 * 4);                    // arrival counter, error flag
  s.total = o;
  return s;
}

}  // namespace
}  // namespace moe

extern "C" size_t moe_schedule_workspace(int64_t N, int32_t L, int32_t E, int32_t k) {
  if (N < 1 || L < 1 || E < 1 || k < 1) return 0;
  return moe::sch_layout(N, L, E, k).total;
}

extern "C" int moe_schedule(const uint8_t* routes, int64_t N, int32_t L, int32_t E, int32_t k,
                            int64_t n1, int32_t max_iters, int32_t keep_original_if_worse,
                            int32_t* perm, int32_t* demand, int64_t* info, void* workspace,
                            size_t ws_bytes, void* stream) {
  using namespace moe;
  MOE_CHECK_ARG(routes && perm && info);
  MOE_CHECK_ARG(N >= 1 && L >= 1 && E >= 1 && E <= 256 && k >= 1 && k <= E);
  MOE_CHECK_ARG(n1 >= 0 && n1 <= N && max_iters >= 1);
  MOE_CHECK_ARG(keep_original_if_worse == 0 || keep_original_if_worse == 1);
  if (N >= ((int64_t)1 << 26) || (int64_t)L * E >= ((int64_t)1 << 24) ||
      (int64_t)L * k >= ((int64_t)1 << 24))
    return MOE_ERR_UNSUPPORTED;
  const SchLayout lay = sch_layout(N, L, E, k);
  if (!workspace || ws_bytes < lay.total || (reinterpret_cast<uintptr_t>(workspace) & 255))
    return MOE_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace);
  auto* bits = reinterpret_cast<uint64_t*>(ws + lay.bits);
  auto* bits_t = reinterpret_cast<uint64_t*>(ws + lay.bits_t);
  auto* ones = reinterpret_cast<int32_t*>(ws + lay.ones);
  auto* rank = reinterpret_cast<int32_t*>(ws + lay.rank);
  auto* order = reinterpret_cast<int32_t*>(ws + lay.order);
  auto* delta = reinterpret_cast<int32_t*>(ws + lay.delta);
  auto* in1 = reinterpret_cast<int32_t*>(ws + lay.in1);
  auto* cnt = reinterpret_cast<int32_t*>(ws + lay.cnt);
  auto* cnt_orig = reinterpret_cast<int32_t*>(ws + lay.cnt_orig);
  auto* hist = reinterpret_cast<int32_t*>(ws + lay.hist);
  auto* tot = reinterpret_cast<unsigned long long*>(ws + lay.tot);
  auto* state = reinterpret_cast<int64_t*>(ws + lay.state);
  auto* cand = reinterpret_cast<Cand*>(ws + lay.cand);
  auto* cand2 = reinterpret_cast<unsigned long long*>(ws + lay.cand2);
  auto* tiecnt = reinterpret_cast<int32_t*>(ws + lay.tiecnt);
  auto* bar = reinterpret_cast<unsigned*>(ws + lay.bar);
  auto* err = reinterpret_cast<int32_t*>(ws + lay.bar + 4);

  const int n = (int)N, W = (L * E + 63) / 64, LE = L * E;
  const int nbins = 4 * L * k + 1, off = 2 * L * k;
  const int nblk = (int)ceil_div(N, kT);
  const size_t cc_lds = (2 * (size_t)LE <= 8192) ? 2 * (size_t)LE * sizeof(int32_t) : 0;
  hipStream_t st = as_stream(stream);
  const dim3 grid(nblk), blk(kT);
#define MOE_TRY(expr) \
  do { if ((expr) != hipSuccess) return MOE_ERR_HIP; } while (0)

  const bool trivial = (n1 == 0 || n1 == N);

  sch_init<<<dim3((unsigned)std::min<int64_t>(64, ceil_div(std::max(nbins, 2 * LE), kT))), blk, 0,
             st>>>(hist, nbins, cnt_orig, 2 * LE, tot, cand2, bar, err, state);
  MOE_CHECK_LAUNCH();
  sch_pack<<<grid, blk, 0, st>>>(routes, n, L, E, k, W, bits, bits_t, ones, rank);
  MOE_CHECK_LAUNCH();
  auto launch_rank = [&]() -> int {
    if (W <= 32) {
      const int tile = std::min(256, 65536 / (8 * W));
      const dim3 g2(nblk, (unsigned)ceil_div(N, tile));
      const size_t lds = (size_t)tile * W * sizeof(uint64_t);
      if (W <= 4) sch_rank_keys<4><<<g2, blk, lds, st>>>(bits, n, W, tile, rank);
      else if (W <= 8) sch_rank_keys<8><<<g2, blk, lds, st>>>(bits, n, W, tile, rank);
      else if (W <= 16) sch_rank_keys<16><<<g2, blk, lds, st>>>(bits, n, W, tile, rank);
      else sch_rank_keys<32><<<g2, blk, lds, st>>>(bits, n, W, tile, rank);
    } else {
      sch_rank<<<dim3(nblk, (unsigned)ceil_div(N, kRankTile)), blk, 0, st>>>(bits, n, W, rank);
    }
    if (hipGetLastError() != hipSuccess) return MOE_ERR_HIP;
    sch_order<<<grid, blk, 0, st>>>(rank, n, order);
    return hipGetLastError() != hipSuccess ? MOE_ERR_HIP : MOE_OK;
  };

  bool done = false;
  const bool coop_fits = LE <= kCoopMaxLE && N < (1 << 24) && 2 * (int64_t)L * k < (1 << 15);
  if (!trivial && coop_fits) {
    const int rc = launch_rank();
    if (rc != MOE_OK) return rc;
    const int cus = device_cu_count();
    const int nb = (int)std::max<int64_t>(1, std::min<int64_t>(cus, ceil_div(N, kCoopT)));
    CoopArgs ca{bits_t, ones, rank, order, n, W, LE, (int)n1, nbins, off, max_iters, 0,
                2 * L * k, delta, in1, hist, cnt, cnt_orig, tot, cand2, tiecnt, bar, err, state};
    void* args[] = {&ca};
    if (hipLaunchCooperativeKernel(reinterpret_cast<const void*>(&sch_coop), dim3(nb),
                                   dim3(kCoopT), args, 0, st) == hipSuccess) {
      done = true;
    } else {
      (void)hipGetLastError();                 // fall back to one launch per phase
      MOE_TRY(fill_i64(state, 0, ST_NWORDS, st));
      MOE_TRY(fill_i32(cnt_orig, 0, 2 * (int64_t)LE, st));
      MOE_TRY(fill_i32(hist, 0, nbins, st));
    }
  }
  if (!done) {
    MOE_TRY(fill_i32(cnt, 0, 2 * (int64_t)LE, st));
    MOE_TRY(fill_i64(reinterpret_cast<int64_t*>(tot), 0, 2, st));
    // Eq. 2 of the input split; the column counts of [0,n1) and [n1,N).
    sch_colcount<<<grid, blk, cc_lds, st>>>(bits, ones, n, W, LE, 1, (int)n1, in1, cnt_orig,
                                           tot, state);
    MOE_CHECK_LAUNCH();
    if (!trivial) {
      MOE_TRY(fill_i64(reinterpret_cast<int64_t*>(tot), 0, 2, st));
      if (!coop_fits) {
        const int rc = launch_rank();
        if (rc != MOE_OK) return rc;
      }
      // m1: least total distance to every token
      sch_colcount<<<grid, blk, cc_lds, st>>>(bits, ones, n, W, LE, 0, (int)n1, in1, cnt, tot,
                                             state);
      MOE_CHECK_LAUNCH();
      sch_cand<<<grid, blk, 0, st>>>(bits, ones, rank, n, W, LE, 0, (int)n1, in1, cnt, tot,
                                     state, cand);
      MOE_CHECK_LAUNCH();
      sch_pick<<<dim3(1), dim3(kSel), 0, st>>>(cand, nblk, 0, state);
      MOE_CHECK_LAUNCH();
      // m2: farthest from m1
      sch_cand<<<grid, blk, 0, st>>>(bits, ones, rank, n, W, LE, 1, (int)n1, in1, cnt, tot,
                                     state, cand);
      MOE_CHECK_LAUNCH();
      sch_pick<<<dim3(1), dim3(kSel), 0, st>>>(cand, nblk, 1, state);
      MOE_CHECK_LAUNCH();
      for (int it = 0; it < max_iters; ++it) {
        sch_delta<<<grid, blk, 0, st>>>(bits, n, W, off, delta, hist, state);
        MOE_CHECK_LAUNCH();
        sch_select<<<dim3(1), dim3(kSel), 0, st>>>(n, (int)n1, nbins, off, delta, order, hist,
                                                  in1, cnt, LE, tot, state);
        MOE_CHECK_LAUNCH();
        sch_colcount<<<grid, blk, cc_lds, st>>>(bits, ones, n, W, LE, 2, (int)n1, in1, cnt, tot,
                                               state);
        MOE_CHECK_LAUNCH();
        sch_cand<<<grid, blk, 0, st>>>(bits, ones, rank, n, W, LE, 2, (int)n1, in1, cnt, tot,
                                       state, cand);
        MOE_CHECK_LAUNCH();
        sch_pick<<<dim3(1), dim3(kSel), 0, st>>>(cand, nblk, 2, state);
        MOE_CHECK_LAUNCH();
      }
    }
  }
  sch_finish<<<dim3(1), dim3(kSel), 0, st>>>(n, (int)n1, L, E, keep_original_if_worse,
                                            trivial ? 1 : 0, in1, cnt, cnt_orig, state, err,
                                            perm, demand, info);
  MOE_CHECK_LAUNCH();
#undef MOE_TRY
  return MOE_OK;
}
