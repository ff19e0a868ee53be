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
         uint64_t* __restrict__ bits, int32_t* __restrict__ ones) {
  const int i = blockIdx.x * kT + threadIdx.x;
  if (i >= N) return;
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
  for (int w = 0; w < W; ++w) c += __popcll(b[w]);
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
    info[0] = trivial ? 0 : state[ST_ITERS];
    info[1] = trivial ? 1 : state[ST_CONV];
    info[2] = trivial ? -1 : state[ST_AM1];
    info[3] = trivial ? -1 : state[ST_AM2];
    info[4] = before;
    info[5] = use_orig ? before : after;
    info[6] = (!trivial && use_orig) ? 1 : 0;
    info[7] = n1;
  }
}

struct SchLayout {
  size_t bits, ones, rank, order, delta, in1, cnt, cnt_orig, hist, tot, state, cand, total;
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
  s.ones = take(N * 4);
  s.rank = take(N * 4);
  s.order = take(N * 4);
  s.delta = take(N * 4);
  s.in1 = take(N * 4);
  s.cnt = take(2 * LE * 4);
  s.cnt_orig = take(2 * LE * 4);
  s.hist = take(nbins * 4);
  s.tot = take(2 * 8);
  s.state = take(ST_NWORDS * 8);
  s.cand = take(nblk * 2 * sizeof(Cand));
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

  const int n = (int)N, W = (L * E + 63) / 64, LE = L * E;
  const int nbins = 4 * L * k + 1, off = 2 * L * k;
  const int nblk = (int)ceil_div(N, kT);
  const size_t cc_lds = (2 * (size_t)LE <= 8192) ? 2 * (size_t)LE * sizeof(int32_t) : 0;
  hipStream_t st = as_stream(stream);
  const dim3 grid(nblk), blk(kT);
#define MOE_TRY(expr) \
  do { if ((expr) != hipSuccess) return MOE_ERR_HIP; } while (0)

  MOE_TRY(fill_i64(state, 0, ST_NWORDS, st));
  MOE_TRY(fill_i32(cnt, 0, 2 * (int64_t)LE, st));
  MOE_TRY(fill_i32(cnt_orig, 0, 2 * (int64_t)LE, st));
  MOE_TRY(fill_i64(reinterpret_cast<int64_t*>(tot), 0, 2, st));
  sch_pack<<<grid, blk, 0, st>>>(routes, n, L, E, k, W, bits, ones);
  MOE_CHECK_LAUNCH();
  // Eq. 2 of the input split; the column counts of [0,n1) and [n1,N).
  unsigned long long* tot_scratch = tot;  // reset by sch_select before reuse
  sch_colcount<<<grid, blk, cc_lds, st>>>(bits, ones, n, W, LE, 1, (int)n1, in1, cnt_orig,
                                         tot_scratch, state);
  MOE_CHECK_LAUNCH();
  const bool trivial = (n1 == 0 || n1 == N);
  if (!trivial) {
    MOE_TRY(fill_i32(rank, 0, N, st));
    MOE_TRY(fill_i32(hist, 0, nbins, st));
    MOE_TRY(fill_i64(reinterpret_cast<int64_t*>(tot), 0, 2, st));
    sch_rank<<<dim3(nblk, (unsigned)ceil_div(N, kRankTile)), blk, 0, st>>>(bits, n, W, rank);
    MOE_CHECK_LAUNCH();
    sch_order<<<grid, blk, 0, st>>>(rank, n, order);
    MOE_CHECK_LAUNCH();
    // m1: least total distance to every token
    sch_colcount<<<grid, blk, cc_lds, st>>>(bits, ones, n, W, LE, 0, (int)n1, in1, cnt, tot,
                                           state);
    MOE_CHECK_LAUNCH();
    sch_cand<<<grid, blk, 0, st>>>(bits, ones, rank, n, W, LE, 0, (int)n1, in1, cnt, tot, state,
                                   cand);
    MOE_CHECK_LAUNCH();
    sch_pick<<<dim3(1), dim3(kSel), 0, st>>>(cand, nblk, 0, state);
    MOE_CHECK_LAUNCH();
    // m2: farthest from m1
    sch_cand<<<grid, blk, 0, st>>>(bits, ones, rank, n, W, LE, 1, (int)n1, in1, cnt, tot, state,
                                   cand);
    MOE_CHECK_LAUNCH();
    sch_pick<<<dim3(1), dim3(kSel), 0, st>>>(cand, nblk, 1, state);
    MOE_CHECK_LAUNCH();
    for (int it = 0; it < max_iters; ++it) {
      sch_delta<<<grid, blk, 0, st>>>(bits, n, W, off, delta, hist, state);
      MOE_CHECK_LAUNCH();
      sch_select<<<dim3(1), dim3(kSel), 0, st>>>(n, (int)n1, nbins, off, delta, order, hist, in1,
                                                cnt, LE, tot, state);
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
  sch_finish<<<dim3(1), dim3(kSel), 0, st>>>(n, (int)n1, L, E, keep_original_if_worse,
                                            trivial ? 1 : 0, in1, cnt, cnt_orig, state, perm,
                                            demand, info);
  MOE_CHECK_LAUNCH();
#undef MOE_TRY
  return MOE_OK;
}
