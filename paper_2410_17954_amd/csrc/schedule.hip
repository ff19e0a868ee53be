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
//            a, so the order is decided word by word on the packed paths: first
//            by counting, for every token, the tokens whose (first word, index)
//            precede its own, then by re-ranking each run of equal first words
//            on the remaining words.
//   init     m1 = argmin_i sum_j d_ij over all tokens, m2 = argmax_i d(i, m1)
//   iterate  delta_i = d(i,m1) - d(i,m2) and its histogram; the threshold
//            delta* where the count reaches n1; batch 1 = delta < delta* plus
//            the first tokens at delta* in signature order; per-batch column
//            counts c_b; sum_{j in C} d_ij = |C| |r_i| + sum_j |r_j|
//            - 2 sum_{b in r_i} c_b; per-batch argmin -> new centroids;
//            a device-side flag stops the remaining rounds once they settle
//   finish   Eq. 2 before/after from the column counts, the optional guard,
//            perm by stable compaction, demand, info.
// All ties go to the lower signature rank. The launch sequence depends only
// on the shapes and max_iters; nothing is read back to the host.
#include "common.h"

#include <algorithm>

namespace moe {
namespace {

constexpr int kT = 256;          // threads of grid-parallel kernels
constexpr int kSel = 1024;       // threads of single-block kernels

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
         uint64_t* __restrict__ bits, uint64_t* __restrict__ bits_t, uint64_t* __restrict__ key0,
         int32_t* __restrict__ ones) {
  const int i = blockIdx.x * kT + threadIdx.x;
  if (i >= N) return;
  const int LE = L * E;
  const uint8_t* r = routes + (int64_t)i * L * k;
  uint64_t* b = bits + (int64_t)i * W;
  int c = 0;
  // Word w holds bits [64w, 64w + 64): only the layers that overlap it are read.
  for (int w = 0; w < W; ++w) {
    const int lo = w * 64, hi = min(lo + 64, LE);
    uint64_t word = 0;
    for (int l = lo / E; l * E < hi; ++l)
      for (int j = 0; j < k; ++j) {
        const int e = r[l * k + j];
        const int bit = l * E + e - lo;
        if (e < E && bit >= 0 && bit < 64) word |= 1ull << bit;
      }
    b[w] = word;
    bits_t[(int64_t)w * N + i] = word;          // word-major copy: coalesced per word
    c += __popcll(word);
    // Signature order on the first word alone is ascending order of the
    // complemented bit reversal: the lowest differing bit becomes the highest.
    if (w == 0) key0[i] = ~__builtin_bitreverse64(word);
  }
  ones[i] = c;
}

// Signature rank, first level: part[t][i] = #{j in j-tile t : (key0_j, j) <
// (key0_i, i)}. The j-keys are uniform across the wave (scalar loads), so a
// pair costs one 64-bit compare and one add with carry; the index tie-break
// is uniform per tile except on the tile that overlaps the block's own rows.
__global__ void __launch_bounds__(kT)
sch_rank_first(const uint64_t* __restrict__ key0, int N, int tile, int32_t* __restrict__ part) {
  const int i = blockIdx.x * kT + threadIdx.x;
  const int j0 = blockIdx.y * tile;
  const int jn = min(tile, N - j0);
  const int ib0 = blockIdx.x * kT, ib1 = min(N, ib0 + kT) - 1;
  const uint64_t ki = i < N ? key0[i] : 0ull;
  const uint64_t* kj = key0 + j0;
  int cnt = 0;
  if (j0 + jn - 1 < ib0) {                          // every j < every i: ties count
    int q = 0;
    for (; q + 16 <= jn; q += 16)
#pragma unroll
      for (int u = 0; u < 16; ++u) cnt += kj[q + u] <= ki;
    for (; q < jn; ++q) cnt += kj[q] <= ki;
  } else if (j0 > ib1) {                            // every j > every i: ties do not
    int q = 0;
    for (; q + 16 <= jn; q += 16)
#pragma unroll
      for (int u = 0; u < 16; ++u) cnt += kj[q + u] < ki;
    for (; q < jn; ++q) cnt += kj[q] < ki;
  } else {
    for (int q = 0; q < jn; ++q) {
      const uint64_t a = kj[q];
      cnt += a < ki || (a == ki && j0 + q < i);
    }
  }
  if (i < N) part[(int64_t)blockIdx.y * N + i] = cnt;
}

// rank[i] = sum of the tile counts; order1[rank[i]] = i.
__global__ void __launch_bounds__(kT)
sch_order_first(const int32_t* __restrict__ part, int ntiles, int N, int32_t* __restrict__ rank,
                int32_t* __restrict__ order1) {
  const int i = blockIdx.x * kT + threadIdx.x;
  if (i >= N) return;
  int r = 0;
  for (int t = 0; t < ntiles; ++t) r += part[(int64_t)t * N + i];
  rank[i] = r;
  order1[r] = i;
}

// Runs of equal first words in first-level order: gs[p] / ge[p] = first / last
// position of the run holding position p. One block; each thread walks a
// contiguous chunk and the chunk boundaries are joined by block scans.
__global__ void __launch_bounds__(kSel)
sch_tie_runs(const uint64_t* __restrict__ key0, const int32_t* __restrict__ order1, int N,
             int32_t* __restrict__ gs, int32_t* __restrict__ ge) {
  __shared__ int s_a[kSel];
  const int tid = threadIdx.x;
  const int per = (N + kSel - 1) / kSel;
  const int p0 = min(N, tid * per), p1 = min(N, p0 + per);
  auto key = [&](int p) { return key0[order1[p]]; };
  // last run start inside the chunk
  int last = -1;
  for (int p = p0; p < p1; ++p)
    if (p == 0 || key(p) != key(p - 1)) last = p;
  s_a[tid] = last;
  __syncthreads();
  for (int o = 1; o < kSel; o <<= 1) {              // inclusive max-scan
    const int v = tid >= o ? s_a[tid - o] : -1;
    __syncthreads();
    s_a[tid] = max(s_a[tid], v);
    __syncthreads();
  }
  int cur = tid > 0 ? s_a[tid - 1] : -1;
  for (int p = p0; p < p1; ++p) {
    if (p == 0 || key(p) != key(p - 1)) cur = p;
    gs[p] = cur;
  }
  __syncthreads();
  // first run end inside the chunk
  int first = N;
  for (int p = p1 - 1; p >= p0; --p)
    if (p == N - 1 || key(p) != key(p + 1)) first = p;
  s_a[tid] = first;
  __syncthreads();
  for (int o = 1; o < kSel; o <<= 1) {              // inclusive min-scan from the right
    const int v = tid + o < kSel ? s_a[tid + o] : N;
    __syncthreads();
    s_a[tid] = min(s_a[tid], v);
    __syncthreads();
  }
  cur = tid + 1 < kSel ? s_a[tid + 1] : N;
  for (int p = p1 - 1; p >= p0; --p) {
    if (p == N - 1 || key(p) != key(p + 1)) cur = p;
    ge[p] = cur;
  }
}

// Second level: inside a run of equal first words the remaining words (then
// the token index) decide; rank[i] = run start + #{run members before i}.
__global__ void __launch_bounds__(kT)
sch_rank_ties(const uint64_t* __restrict__ bits, int N, int W, const int32_t* __restrict__ order1,
              const int32_t* __restrict__ gs, const int32_t* __restrict__ ge,
              int32_t* __restrict__ rank) {
  const int p = blockIdx.x * kT + threadIdx.x;
  if (p >= N) return;
  const int s = gs[p], e = ge[p];
  if (s == e) return;
  const int i = order1[p];
  const uint64_t* bi = bits + (int64_t)i * W;
  int cnt = 0;
  for (int m = s; m <= e; ++m) {
    if (m == p) continue;
    const int j = order1[m];
    const uint64_t* bj = bits + (int64_t)j * W;
    int before = j < i;
    for (int w = 1; w < W; ++w) {
      const uint64_t a = bj[w];
      const uint64_t d = a ^ bi[w];
      if (d) {
        before = (a & lowbit(d)) != 0;
        break;
      }
    }
    cnt += before;
  }
  rank[i] = s + cnt;
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
  size_t bits, bits_t, key0, ones, rank, part, order1, runs, order, delta, in1, cnt, cnt_orig,
      hist, tot, state, cand, cand2, tiecnt, bar, total;
};

// j-tiling of the first-level rank: about 2048 blocks in all, tiles of a
// multiple of 64 tokens.
struct RankTiles {
  int tile, ntiles;
};

RankTiles rank_tiles(int64_t N) {
  const int64_t nbi = ceil_div(N, kT);
  const int64_t want = std::max<int64_t>(1, std::min<int64_t>(64, 2048 / nbi));
  const int64_t tile = align_up(ceil_div(N, want), 64);
  return RankTiles{(int)tile, (int)ceil_div(N, tile)};
}

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
  s.key0 = take(N * 8);
  s.ones = take(N * 4);
  s.rank = take(N * 4);
  s.part = take((size_t)rank_tiles(N).ntiles * N * 4);
  s.order1 = take(N * 4);
  s.runs = take(2 * N * 4);
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
  auto* key0 = reinterpret_cast<uint64_t*>(ws + lay.key0);
  auto* part = reinterpret_cast<int32_t*>(ws + lay.part);
  auto* order1 = reinterpret_cast<int32_t*>(ws + lay.order1);
  auto* run_s = reinterpret_cast<int32_t*>(ws + lay.runs);
  auto* run_e = run_s + N;
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
  sch_pack<<<grid, blk, 0, st>>>(routes, n, L, E, k, W, bits, bits_t, key0, ones);
  MOE_CHECK_LAUNCH();
  // Signature order: (first word, index) by counting, then runs of equal
  // first words re-ranked on the remaining words.
  auto launch_rank = [&]() -> int {
    const RankTiles rt = rank_tiles(N);
    sch_rank_first<<<dim3(nblk, rt.ntiles), blk, 0, st>>>(key0, n, rt.tile, part);
    if (hipGetLastError() != hipSuccess) return MOE_ERR_HIP;
    sch_order_first<<<grid, blk, 0, st>>>(part, rt.ntiles, n, rank, W > 1 ? order1 : order);
    if (hipGetLastError() != hipSuccess) return MOE_ERR_HIP;
    if (W > 1) {
      sch_tie_runs<<<dim3(1), dim3(kSel), 0, st>>>(key0, order1, n, run_s, run_e);
      if (hipGetLastError() != hipSuccess) return MOE_ERR_HIP;
      sch_rank_ties<<<grid, blk, 0, st>>>(bits, n, W, order1, run_s, run_e, rank);
      if (hipGetLastError() != hipSuccess) return MOE_ERR_HIP;
      sch_order<<<grid, blk, 0, st>>>(rank, n, order);
      if (hipGetLastError() != hipSuccess) return MOE_ERR_HIP;
    }
    return MOE_OK;
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
