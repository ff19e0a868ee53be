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
//            a, which for one word is descending order of its bit reversal.
//            Chunks of 512 tokens are sorted in LDS (bitonic) on the first three
//            words, later words and the index deciding ties; the signature rank
//            of a token is the sum of its lower bounds in every sorted chunk.
//   init     m1 = argmin_i sum_j d_ij over all tokens, m2 = argmax_i d(i, m1)
//   iterate  delta_i = d(i,m1) - d(i,m2) and its histogram; the threshold
//            delta* where the count reaches n1; batch 1 = delta < delta* plus
//            the first tokens at delta* in signature order; per-batch column
//            counts c_b; sum_{j in C} d_ij = |C| |r_i| + sum_j |r_j|
//            - 2 sum_{b in r_i} c_b; per-batch argmin -> new centroids, until
//            they repeat or max_iters rounds
//   finish   Eq. 2 before/after from the column counts, the optional guard,
//            perm by stable compaction, demand, info.
// All ties go to the lower signature rank. Up to 1024 tokens whose paths fit
// in LDS run every step in one block (sch_small); otherwise the rounds run in
// one resident-grid launch over tokens laid out in signature order (a per-phase
// launch sequence covers shapes beyond its limits). Nothing is read back to
// the host.
#include "common.h"

#include <algorithm>
#include <vector>

namespace moe {
namespace {

constexpr int kT = 256;          // threads of grid-parallel kernels
constexpr int kSel = 1024;       // threads of single-block and finish kernels
constexpr int kPackT = 64;       // tokens per pack block
constexpr int kPackMaxBytes = 16384;  // route bytes a pack block stages in LDS
constexpr int kChunk = 512;      // tokens per sorted chunk
constexpr int kSortT = 256;      // threads of the chunk sort blocks
constexpr int kMergeT = 1024;    // threads of the merge-rank blocks
constexpr int kMaxRankGroups = 16;    // chunk groups of the merge rank

// state words
enum {
  ST_M1 = 0, ST_M2, ST_DONE, ST_ITERS, ST_CONV, ST_AM1, ST_AM2, ST_USE_ORIG, ST_BEFORE,
  ST_AFTER, ST_NWORDS = 16
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
// Packs kPackT tokens per block: their routes are staged in LDS with
// coalesced loads when they fit, each token's words are built in registers
// (only the layers overlapping a word are read for it) and written row-major.
// key0 / key1 / key2 are the sort keys of the first three words (0 past W).
template <bool STAGED>
__global__ void __launch_bounds__(kPackT)
sch_pack(const uint8_t* __restrict__ routes, int N, int L, int E, int k, int W,
         uint64_t* __restrict__ bits, uint64_t* __restrict__ key0, uint64_t* __restrict__ key1,
         uint64_t* __restrict__ key2, int32_t* __restrict__ ones) {
  __shared__ __attribute__((aligned(16))) uint8_t s_r[kPackMaxBytes];
  const int Lk = L * k, LE = L * E;
  const int t0 = blockIdx.x * kPackT;
  const int nt = min(kPackT, N - t0);
  const uint8_t* src = routes + (int64_t)t0 * Lk;
  if constexpr (STAGED) {
    // 16-byte pieces, eight loads in flight per thread, then the odd tail
    const int nbytes = nt * Lk;
    int q0 = 0;
    if ((reinterpret_cast<uintptr_t>(src) & 15) == 0) {
      const uint4* s16 = reinterpret_cast<const uint4*>(src);
      uint4* d16 = reinterpret_cast<uint4*>(s_r);
      const int n16 = nbytes / 16;
      for (int q = threadIdx.x; q < n16; q += 8 * kPackT) {
        uint4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (q + u * kPackT < n16) v[u] = s16[q + u * kPackT];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (q + u * kPackT < n16) d16[q + u * kPackT] = v[u];
      }
      q0 = n16 * 16;
    }
    for (int q = q0 + threadIdx.x; q < nbytes; q += kPackT) s_r[q] = src[q];
    __syncthreads();
  }
  const int t = threadIdx.x;
  if (t >= nt) return;
  const int i = t0 + t;
  const uint8_t* r;
  if constexpr (STAGED) r = s_r + t * Lk;
  else r = src + (int64_t)t * Lk;
  uint64_t* b = bits + (int64_t)i * W;
  uint64_t k0 = 0, k1 = 0, k2 = 0;
  int c = 0;
  for (int w = 0; w < W; ++w) {
    const int lo = w * 64, hi = min(lo + 64, LE);
    uint64_t word = 0;
    for (int l = lo / E; l * E < hi; ++l) {
      auto set = [&](int e) {
        const int bit = l * E + e - lo;
        if (e < E && bit >= 0 && bit < 64) word |= 1ull << bit;
      };
      if (k <= 8) {                              // the layer's ids read together
        int ev[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) ev[j] = j < k ? r[l * k + j] : E;
#pragma unroll
        for (int j = 0; j < 8; ++j) set(ev[j]);
      } else {
        for (int j = 0; j < k; ++j) set(r[l * k + j]);
      }
    }
    b[w] = word;
    c += __popcll(word);
    if (w == 0) k0 = ~__builtin_bitreverse64(word);
    if (w == 1) k1 = ~__builtin_bitreverse64(word);
    if (w == 2) k2 = ~__builtin_bitreverse64(word);
  }
  key0[i] = k0;
  key1[i] = k1;
  key2[i] = k2;
  ones[i] = c;
}

// (key0, key1, key2, token) order; when the first three words agree, the
// later words of the packed paths decide (lowest differing bit set first),
// then the token index. Indices >= N are padding and compare by index alone.
struct SKey {
  uint64_t k0, k1, k2;
  int32_t idx;
};
__device__ __forceinline__ bool key_less(const SKey& a, const SKey& b,
                                         const uint64_t* __restrict__ bits, int W, int N) {
  if (a.k0 != b.k0) return a.k0 < b.k0;
  if (a.k1 != b.k1) return a.k1 < b.k1;
  if (a.k2 != b.k2) return a.k2 < b.k2;
  const int ia = a.idx, ib = b.idx;
  if (ia == ib) return false;                    // a token against itself
  if (W > 3 && ia < N && ib < N) {
    // eight words of each path per round trip
    const uint64_t* pa = bits + (int64_t)ia * W;
    const uint64_t* pb = bits + (int64_t)ib * W;
    for (int w0 = 3; w0 < W; w0 += 8) {
      uint64_t va[8], vb[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        va[u] = w0 + u < W ? pa[w0 + u] : 0ull;
        vb[u] = w0 + u < W ? pb[w0 + u] : 0ull;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint64_t d = va[u] ^ vb[u];
        if (d) return (va[u] & lowbit(d)) != 0;
      }
    }
  }
  return ia < ib;
}

// Sorts each chunk of kChunk consecutive tokens by key_less (bitonic network
// in LDS, one compare-exchange per thread and step; the tail chunk is padded
// with keys that sort last).
__global__ void __launch_bounds__(kSortT)
sch_sort_chunks(const uint64_t* __restrict__ key0, const uint64_t* __restrict__ key1,
                const uint64_t* __restrict__ key2, const uint64_t* __restrict__ bits, int N,
                int W, uint64_t* __restrict__ s0, uint64_t* __restrict__ s1,
                uint64_t* __restrict__ s2, int32_t* __restrict__ sidx) {
  static_assert(kChunk == 2 * kSortT, "one compare-exchange per thread and step");
  __shared__ uint64_t a0[kChunk], a1[kChunk], a2[kChunk];
  __shared__ int32_t ai[kChunk];
  const int c0 = blockIdx.x * kChunk;
  const int cn = min(kChunk, N - c0);
  for (int p = threadIdx.x; p < kChunk; p += kSortT) {
    const bool real = p < cn;
    a0[p] = real ? key0[c0 + p] : ~0ull;
    a1[p] = real ? key1[c0 + p] : ~0ull;
    a2[p] = real ? key2[c0 + p] : ~0ull;
    ai[p] = real ? c0 + p : INT32_MAX;
  }
  __syncthreads();
  const int t = threadIdx.x;
  for (int kk = 2; kk <= kChunk; kk <<= 1) {
    for (int j = kk >> 1; j > 0; j >>= 1) {
      const int x = ((t & ~(j - 1)) << 1) | (t & (j - 1));   // bit j of x clear
      const int y = x + j;
      const bool up = (x & kk) == 0;
      const SKey kx{a0[x], a1[x], a2[x], ai[x]}, ky{a0[y], a1[y], a2[y], ai[y]};
      if (key_less(ky, kx, bits, W, N) == up) {    // pairs are disjoint within a step
        a0[x] = ky.k0; a1[x] = ky.k1; a2[x] = ky.k2; ai[x] = ky.idx;
        a0[y] = kx.k0; a1[y] = kx.k1; a2[y] = kx.k2; ai[y] = kx.idx;
      }
      __syncthreads();
    }
  }
  for (int p = threadIdx.x; p < cn; p += kSortT) {
    s0[c0 + p] = a0[p];
    s1[c0 + p] = a1[p];
    s2[c0 + p] = a2[p];
    sidx[c0 + p] = ai[p];
  }
}

// part[g][i] = #{tokens before i} summed over the sorted chunks of group g
// (chunks g, g + G, g + 2G, ...): each chunk is staged in LDS and searched
// with a branch-free lower bound.
__global__ void __launch_bounds__(kMergeT)
sch_merge_rank(const uint64_t* __restrict__ key0, const uint64_t* __restrict__ key1,
               const uint64_t* __restrict__ key2, const uint64_t* __restrict__ bits, int N,
               int W, int nchunks, const uint64_t* __restrict__ s0,
               const uint64_t* __restrict__ s1, const uint64_t* __restrict__ s2,
               const int32_t* __restrict__ sidx, int32_t* __restrict__ part) {
  __shared__ uint64_t a0[kChunk], a1[kChunk], a2[kChunk];
  __shared__ int32_t ai[kChunk];
  const int i = blockIdx.x * kMergeT + threadIdx.x;
  const SKey me{i < N ? key0[i] : 0ull, i < N ? key1[i] : 0ull, i < N ? key2[i] : 0ull, i};
  int cnt = 0;
  for (int c = blockIdx.y; c < nchunks; c += gridDim.y) {
    const int c0 = c * kChunk;
    const int cn = min(kChunk, N - c0);
    __syncthreads();
    for (int p = threadIdx.x; p < cn; p += kMergeT) {
      a0[p] = s0[c0 + p];
      a1[p] = s1[c0 + p];
      a2[p] = s2[c0 + p];
      ai[p] = sidx[c0 + p];
    }
    __syncthreads();
    if (i < N) {
      int lo = 0;
      for (int step = kChunk; step > 0; step >>= 1) {
        const int m = lo + step - 1;
        if (lo + step <= cn && key_less(SKey{a0[m], a1[m], a2[m], ai[m]}, me, bits, W, N))
          lo += step;
      }
      cnt += lo;
    }
  }
  if (i < N) part[(int64_t)blockIdx.y * N + i] = cnt;
}

// rank[i] = sum over groups; order[rank[i]] = i.
__global__ void __launch_bounds__(kT)
sch_rank_sum(const int32_t* __restrict__ part, int ngroups, int N, int32_t* __restrict__ rank,
             int32_t* __restrict__ order) {
  const int i = blockIdx.x * kT + threadIdx.x;
  if (i >= N) return;
  int r = 0;
  for (int g = 0; g < ngroups; ++g) r += part[(int64_t)g * N + i];
  rank[i] = r;
  if (r < N) order[r] = i;                        // always: the chunk counts add up to a permutation
}

// Merge passes for large N (the rank above costs N lower bounds per chunk):
// sorted runs of R tokens become runs of 2R. Block b writes outputs
// [b T, b T + T) of the pass, T = min(kMergeTile, 2R) so that a block stays
// inside one pair of runs. Two threads find where the block's first and
// one-past-last outputs split the pair (merge path: a binary search along the
// diagonal), the two pieces are staged in LDS, and each thread merges T / 256
// consecutive outputs after the same search inside LDS.
constexpr int kMergeTile = 2048;
constexpr int kMergeBT = 256;
constexpr int kMergeRankMaxChunks = 256;         // beyond: merge passes

__device__ __forceinline__ SKey skey_at(const uint64_t* __restrict__ s0,
                                        const uint64_t* __restrict__ s1,
                                        const uint64_t* __restrict__ s2,
                                        const int32_t* __restrict__ si, int64_t p) {
  return SKey{s0[p], s1[p], s2[p], si[p]};
}

__global__ void __launch_bounds__(kMergeBT)
sch_merge_pass(const uint64_t* __restrict__ s0, const uint64_t* __restrict__ s1,
               const uint64_t* __restrict__ s2, const int32_t* __restrict__ si,
               const uint64_t* __restrict__ bits, int N, int W, int R, uint64_t* __restrict__ d0,
               uint64_t* __restrict__ d1, uint64_t* __restrict__ d2, int32_t* __restrict__ di) {
  __shared__ uint64_t a0[kMergeTile], a1[kMergeTile], a2[kMergeTile];
  __shared__ int32_t ai[kMergeTile];
  __shared__ int32_t s_src[kMergeTile];          // merged order: staged position per output
  __shared__ int s_lo[2], s_hi[2], s_cut[2];
  const int tid = threadIdx.x;
  const int T = min(kMergeTile, 2 * R);
  const int o0 = blockIdx.x * T;                 // first output of the block
  const int ps = o0 / (2 * R) * (2 * R);         // the pair's first position
  const int nA = min(R, N - ps);
  const int nB = max(0, min(R, N - ps - R));
  const int aS = ps, bS = ps + nA;
  const int dbeg = o0 - ps, dend = min(dbeg + T, nA + nB);
  // The split of diagonal d is the first a in [max(0, d - nB), min(d, nA)]
  // with !(A[a] < B[d - 1 - a]) (the end if none). Threads 0..127 search
  // diagonal dbeg, 128..255 dend: each round probes 128 evenly spaced a and
  // keeps the gap between the last true and the first false probe.
  static_assert(kMergeBT == 256, "two groups of 128 probes");
  if (tid < 2) {
    const int d = tid ? dend : dbeg;
    s_lo[tid] = max(0, d - nB);
    s_hi[tid] = min(d, nA);
  }
  __syncthreads();
  const int g = tid >> 7, t = tid & 127;
  const int dg = g ? dend : dbeg;
  while (s_lo[0] < s_hi[0] || s_lo[1] < s_hi[1]) {   // the same values in every thread
    const int lo = s_lo[g], hi = s_hi[g], len = hi - lo;
    if (tid < 2) s_cut[tid] = 128;
    __syncthreads();
    if (len > 0) {
      const int a = lo + (int)(((int64_t)t * len) >> 7);
      if (!key_less(skey_at(s0, s1, s2, si, aS + a), skey_at(s0, s1, s2, si, bS + dg - 1 - a),
                    bits, W, N))
        atomicMin(&s_cut[g], t);
    }
    __syncthreads();
    if (len > 0 && t == 0) {
      const int c = s_cut[g];
      s_lo[g] = c == 0 ? lo : lo + (int)(((int64_t)(c - 1) * len) >> 7) + 1;
      s_hi[g] = c == 128 ? hi : lo + (int)(((int64_t)c * len) >> 7);
    }
    __syncthreads();
  }
  const int ja0 = s_lo[0];
  const int na = s_lo[1] - ja0;                  // A elements in the tile, then B
  const int tot = dend - dbeg;
  const int nb = tot - na;
  const int jb0 = dbeg - ja0;
  for (int p = threadIdx.x; p < tot; p += kMergeBT) {
    const int g = p < na ? aS + ja0 + p : bS + jb0 + (p - na);
    a0[p] = s0[g];
    a1[p] = s1[g];
    a2[p] = s2[g];
    ai[p] = si[g];
  }
  __syncthreads();
  auto at = [&](int p) { return SKey{a0[p], a1[p], a2[p], ai[p]}; };
  const int per = T / kMergeBT;
  const int t0 = threadIdx.x * per;
  if (t0 < tot) {
    int lo = max(0, t0 - nb), hi = min(t0, na);
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (key_less(at(mid), at(na + t0 - 1 - mid), bits, W, N))
        lo = mid + 1;
      else
        hi = mid;
    }
    int ia = lo, ib = t0 - lo;
    for (int u = 0; u < per && t0 + u < tot; ++u) {
      const bool take_a = ib >= nb || (ia < na && key_less(at(ia), at(na + ib), bits, W, N));
      s_src[t0 + u] = take_a ? ia++ : na + ib++;
    }
  }
  __syncthreads();
  // the tile's outputs in order: coalesced stores
  for (int p = threadIdx.x; p < tot; p += kMergeBT) {
    const int src = s_src[p];
    d0[o0 + p] = a0[src];
    d1[o0 + p] = a1[src];
    d2[o0 + p] = a2[src];
    di[o0 + p] = ai[src];
  }
}

// rank[order[r]] = r from the fully sorted token ids.
__global__ void __launch_bounds__(kT)
sch_rank_sorted(const int32_t* __restrict__ sorted, int N, int32_t* __restrict__ rank,
                int32_t* __restrict__ order) {
  const int r = blockIdx.x * kT + threadIdx.x;
  if (r >= N) return;
  const int i = sorted[r];
  order[r] = i;
  rank[i] = r;
}

// Paths and path sizes in signature order, word-major: bits_s[w][r] is word w
// of the token at signature position r.
__global__ void __launch_bounds__(kT)
sch_repack(const uint64_t* __restrict__ bits, const int32_t* __restrict__ ones,
           const int32_t* __restrict__ order, int N, int W, uint64_t* __restrict__ bits_s,
           int32_t* __restrict__ ones_s) {
  const int r = blockIdx.x * kT + threadIdx.x;
  if (r >= N) return;
  const int i = order[r];
  const uint64_t* b = bits + (int64_t)i * W;
  for (int w = 0; w < W; ++w) bits_s[(int64_t)w * N + r] = b[w];
  ones_s[r] = ones[i];
}

// ------------------------------------------- per-phase launches (fallback)
// Used when the shapes exceed the round-loop kernel's LDS limits or its
// launch is refused; token-index space throughout.
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

// ------------------------------------------------ resident-grid round loop
// All rounds in one launch whose blocks are all resident at once (at most one
// block per compute unit is needed). Tokens are
// addressed by signature position r: block b owns a contiguous range of at
// most PPT * kCoopT positions, thread t positions t0 + t + j kCoopT (j < PPT),
// and keeps their state (delta, batch) in registers and their path words in
// LDS when they fit, so ties are broken by position directly. Data that
// crosses blocks is written with device-scope atomics (sums, minima) or
// agent-scope atomic stores and read with agent-scope atomic loads -- never
// with plain accesses, since the XCD L2s are not coherent with each other --
// and phases are separated by a grid barrier on a monotonic arrival counter
// that orders those operations (see grid_sync). Every barrier wait
// is bounded: past the bound the block records an error and goes on, so the
// launch always terminates (the result is then flagged, never trusted).
// Candidates are packed as (value << 24 | position); their minimum keeps the
// lower-position tie rule. A round needs three
// barriers: after the histogram, after the assignment, after the candidates.
constexpr int kCoopT = 256;
constexpr int kCoopMaxLE = 8192;
constexpr int kCoopMaxBins = 4096;
constexpr int kCoopMaxBlocks = 1024;
constexpr int kCoopMaxPPT = 16;
constexpr size_t kCoopMaxLds = 160 * 1024 - 2048;   // dynamic LDS limit (static part aside)
constexpr unsigned kSpinBound = 1u << 20;

__device__ __forceinline__ int ld_ag(const int32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned ld_ag(const unsigned* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long ld_ag64(const unsigned long long* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_ag(int32_t* p, int32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_ag64(unsigned long long* p, unsigned long long v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ void grid_sync(unsigned* bar, unsigned nblk, int32_t* err) {
  // Every datum that crosses blocks inside the launch is read and written with
  // agent-scope atomic operations, which are performed coherently across the
  // XCDs (they bypass the XCD-local caches), so the barrier only has to order
  // them: each wave waits until its own memory operations have completed, then
  // one thread arrives and polls. No cache write-back or invalidation is
  // needed -- those cost a serialised L2 operation per wave and block.
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  // One block (a few hundred tokens): the block barrier is the whole barrier;
  // the arrival counter is never touched, so every call takes this branch.
  if (nblk == 1) return;
  if (threadIdx.x == 0) {
    const unsigned arrived = atomicAdd(bar, 1u) + 1u;
    const unsigned target = (arrived + nblk - 1u) / nblk * nblk;
    unsigned spins = 0;
    while (ld_ag(bar) < target) {
      __builtin_amdgcn_s_sleep(1);
      if (++spins == kSpinBound) {
        atomicExch(err, 1);
        break;
      }
    }
  }
  __syncthreads();
}

__device__ __forceinline__ unsigned long long wave_min_u64(unsigned long long v) {
  for (int o = 32; o > 0; o >>= 1) {
    const unsigned long long w = __shfl_xor(v, o, kWave);
    v = w < v ? w : v;
  }
  return v;
}

struct CoopArgs {
  const uint64_t* bits_s;   // [W][N] paths in signature order
  const int32_t* ones_s;    // [N] path sizes in signature order
  const int32_t* order;     // [N] token at each signature position
  const uint8_t* routes;    // [N][L k] route ids by token
  int N, W, LE, n1, nbins, off, max_iters, twoLk, bits_lds, rt_lds, E, k, Lk, L;
  int32_t* in1;             // [N] by token: the final batch-1 flags
  int32_t* hist;            // [2][nbins] global histograms of alternate rounds
  int32_t* hpart;           // [gridDim][nbins] per-block histograms
  int32_t* cnt;             // [LE] batch-1 column counts
  int32_t* cnt_orig;        // [2][LE] column counts of the input split
  unsigned long long* tot;  // [4]: [0] batch-1 path-size sum, [2..3] input split
  unsigned long long* cand; // [4][2][gridDim]: per-block candidates, 3 round slots + start
  unsigned* bar;
  int32_t* err;
  int64_t* state;
};

// Dynamic LDS of the cooperative kernel: the two medoids' words (2 W), the
// block's own path words (PPT W kCoopT) when bits_lds and route ids
// (PPT L k kCoopT bytes) when rt_lds, batch counts (2 LE), all-token counts
// (LE), histogram (nbins).
struct CoopLds {
  size_t c, all, h, med, bits, rt, cb, total;
};
__host__ __device__ inline CoopLds coop_lds(int LE, int nbins, int W, int Lk, int ppt,
                                           bool bits_lds, bool rt_lds) {
  CoopLds s{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = (o + bytes + 15) / 16 * 16;
    return at;
  };
  s.med = take(2 * (size_t)W * 8);
  s.bits = take(bits_lds ? (size_t)ppt * W * kCoopT * 8 : 0);
  s.rt = take(rt_lds ? (size_t)ppt * Lk * kCoopT : 0);
  s.cb = take(rt_lds ? (size_t)Lk * 4 : 0);
  s.c = take(2 * (size_t)LE * 4);
  s.all = take((size_t)LE * 4);
  s.h = take((size_t)nbins * 4);
  s.total = o;
  return s;
}

template <int PPT>
__global__ void __launch_bounds__(kCoopT)
sch_coop(CoopArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ unsigned long long s_red[kCoopT / kWave];
  __shared__ unsigned long long s_tot[2];
  __shared__ int s_thr, s_q;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const unsigned nblk = gridDim.x;
  const int N = a.N, W = a.W, LE = a.LE, nbins = a.nbins, off = a.off, n1 = a.n1;
  const bool bits_lds = a.bits_lds != 0, rt_lds = a.rt_lds != 0;
  const int Lk = a.Lk;
  const CoopLds L = coop_lds(LE, nbins, W, Lk, PPT, bits_lds, rt_lds);
  int32_t* s_c = reinterpret_cast<int32_t*>(smem + L.c);
  int32_t* s_all = reinterpret_cast<int32_t*>(smem + L.all);
  int32_t* s_h = reinterpret_cast<int32_t*>(smem + L.h);
  uint64_t* s_med = reinterpret_cast<uint64_t*>(smem + L.med);      // [2][W]
  uint64_t* s_bits = reinterpret_cast<uint64_t*>(smem + L.bits);    // [PPT][W][kCoopT]
  uint8_t* s_rt = reinterpret_cast<uint8_t*>(smem + L.rt);          // [PPT][L k][kCoopT]
  int32_t* s_cb = reinterpret_cast<int32_t*>(smem + L.cb);          // [L k] first column of the id's layer
  const int per = (N + (int)nblk - 1) / (int)nblk;
  const int t0 = min(N, (int)blockIdx.x * per), t1 = min(N, t0 + per);
  int pos[PPT];
  bool own[PPT];
#pragma unroll
  for (int j = 0; j < PPT; ++j) {
    pos[j] = t0 + tid + j * kCoopT;
    own[j] = pos[j] < t1;
  }

  auto gword = [&](int r, int w) { return a.bits_s[(int64_t)w * N + r]; };
  auto word = [&](int j, int w) {
    return bits_lds ? s_bits[((int64_t)j * W + w) * kCoopT + tid] : gword(pos[j], w);
  };
  const int rot0 = rt_lds ? (lane % a.L) * a.k : 0;
  // The columns of a path: from its route ids staged in LDS (a loop of fixed
  // length L k, ids >= E skipped), else from the set bits of its words.
  auto for_cols = [&](int j, auto&& f) {
    if (rt_lds) {
      // Eight ids per round trip, every access unconditional (clamped index,
      // masked use) so that the loads issue back to back. Lane l starts at
      // layer l mod L: neighbouring positions hold similar routes, and their
      // LDS atomics would otherwise hit the same column together.
      const uint8_t* rt = s_rt + (int64_t)j * Lk * kCoopT + tid;
      int q = rot0;
      for (int q0 = 0; q0 < Lk; q0 += 8) {
        int e[8], base[8];
        bool in[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          in[u] = q0 + u < Lk;
          const int qq = q + u < Lk ? q + u : q + u - Lk;
          const int qc = in[u] ? qq : 0;
          e[u] = rt[qc * kCoopT];
          base[u] = s_cb[qc];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const bool ok = in[u] && e[u] < a.E;
          f(ok ? base[u] + e[u] : 0, ok);
        }
        q += 8;
        q -= q >= Lk ? Lk : 0;
      }
    } else {
      for (int w = 0; w < W; ++w) {
        uint64_t x = word(j, w);
        while (x) {
          f(w * 64 + __builtin_ctzll(x), true);
          x &= x - 1;
        }
      }
    }
  };
  if (bits_lds) {                                // eight words per round trip
#pragma unroll
    for (int j = 0; j < PPT; ++j)
      for (int w0 = 0; w0 < W; w0 += 8) {
        uint64_t v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = (own[j] && w0 + u < W) ? gword(pos[j], w0 + u) : 0ull;
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (w0 + u < W) s_bits[((int64_t)j * W + w0 + u) * kCoopT + tid] = v[u];
      }
  }
  if (rt_lds) {                                  // each token's ids, transposed
    for (int q = tid; q < Lk; q += kCoopT) s_cb[q] = (q / a.k) * a.E;
#pragma unroll
    for (int j = 0; j < PPT; ++j) {
      const uint8_t* src = own[j] ? a.routes + (int64_t)a.order[pos[j]] * Lk : nullptr;
      uint8_t* dst = s_rt + (int64_t)j * Lk * kCoopT + tid;
      if ((Lk & 3) == 0 && (reinterpret_cast<uintptr_t>(a.routes) & 3) == 0) {
        for (int q0 = 0; q0 < Lk; q0 += 32) {        // eight 4-byte loads per round trip
          uint32_t v[8];
#pragma unroll
          for (int u = 0; u < 8; ++u)
            v[u] = (src && q0 + 4 * u < Lk) ? *reinterpret_cast<const uint32_t*>(src + q0 + 4 * u) : 0xFFFFFFFFu;
#pragma unroll
          for (int u = 0; u < 8; ++u)
            if (q0 + 4 * u < Lk)
#pragma unroll
              for (int b = 0; b < 4; ++b) dst[(q0 + 4 * u + b) * kCoopT] = (uint8_t)(v[u] >> (8 * b));
        }
      } else {
        for (int q = 0; q < Lk; ++q) dst[q * kCoopT] = src ? src[q] : 0xFF;
      }
    }
  }
  int ones[PPT];
#pragma unroll
  for (int j = 0; j < PPT; ++j) ones[j] = own[j] ? a.ones_s[pos[j]] : 0;

  auto block_min_u64 = [&](unsigned long long v) {
    v = wave_min_u64(v);
    if (lane == 0) s_red[tid / kWave] = v;
    __syncthreads();
    unsigned long long r = s_red[0];
    for (int w = 1; w < kCoopT / kWave; ++w) r = s_red[w] < r ? s_red[w] : r;
    __syncthreads();
    return r;
  };
  // Candidates: every block stores its minimum in its own entry of a slot
  // (no contended atomics); after the barrier every block reduces the slot.
  auto cand_slot = [&](int slot, int c) { return a.cand + ((int64_t)slot * 2 + c) * nblk; };
  auto put_cand = [&](int slot, int c, unsigned long long v) {
    if (tid == 0) st_ag64(cand_slot(slot, c) + blockIdx.x, v);
  };
  auto min_cand = [&](int slot, int c) {
    const unsigned long long* p = cand_slot(slot, c);
    unsigned long long v = ~0ull;
    for (int b = tid; b < (int)nblk; b += kCoopT) {
      const unsigned long long x = ld_ag64(p + b);
      v = x < v ? x : v;
    }
    return block_min_u64(v);
  };

  // sum of cc over the set bits of x, four gathers in flight (absent bits
  // read cc[0] and add nothing)
  auto gather = [](uint64_t x, const int32_t* cc) -> int {
    int g = 0;
    while (x) {
      int b[4];
      bool has[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        has[u] = x != 0;
        b[u] = has[u] ? __builtin_ctzll(x) : 0;
        x &= x - 1;
      }
      int v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = cc[b[u]];
#pragma unroll
      for (int u = 0; u < 4; ++u) g += has[u] ? v[u] : 0;
    }
    return g;
  };
  // (sum_j in batch d(r, j)) << 24 | r under the counts cc of that batch
  auto dist_key = [&](int j, const int32_t* cc, int64_t size, unsigned long long tot) {
    int64_t g = 0;
    if (rt_lds) {
      int gi = 0;
      for_cols(j, [&](int col, bool ok) {
        const int v = cc[col];
        gi += ok ? v : 0;
      });
      g = gi;
    } else {
      for (int w = 0; w < W; ++w) g += gather(word(j, w), cc + w * 64);
    }
    const int64_t D = size * ones[j] + (int64_t)tot - 2 * g;
    return ((unsigned long long)D << 24) | (unsigned long long)pos[j];
  };
  auto decode = [&](unsigned long long key) {
    const int r = (int)(key & 0xFFFFFF);
    return r < N ? r : 0;                         // empty batch only after a barrier error
  };

  // ---- input split: column counts (Eq. 2 before, demand of the original)
  for (int q = tid; q < 2 * LE; q += kCoopT) s_c[q] = 0;
  if (tid < 2) s_tot[tid] = 0;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < PPT; ++j) {
    if (!own[j]) continue;
    const int c = a.order[pos[j]] < n1 ? 0 : 1;
    int32_t* dst = s_c + c * LE;
    for_cols(j, [&](int col, bool ok) { atomicAdd(&dst[col], ok ? 1 : 0); });
    atomicAdd(&s_tot[c], (unsigned long long)ones[j]);
  }
  __syncthreads();
  for (int q = tid; q < 2 * LE; q += kCoopT)
    if (s_c[q]) atomicAdd(&a.cnt_orig[q], s_c[q]);
  if (tid < 2 && s_tot[tid]) atomicAdd(&a.tot[2 + tid], s_tot[tid]);
  grid_sync(a.bar, nblk, a.err);

  // ---- m1: least total distance; counts over everyone = both input batches
  for (int q = tid; q < LE; q += kCoopT) s_all[q] = ld_ag(a.cnt_orig + q) + ld_ag(a.cnt_orig + LE + q);
  const unsigned long long tot_all = ld_ag64(a.tot + 2) + ld_ag64(a.tot + 3);
  __syncthreads();
  {
    unsigned long long best = ~0ull;
#pragma unroll
    for (int j = 0; j < PPT; ++j) {
      if (!own[j]) continue;
      const unsigned long long key = dist_key(j, s_all, N, tot_all);
      best = key < best ? key : best;
    }
    put_cand(3, 0, block_min_u64(best));
  }
  grid_sync(a.bar, nblk, a.err);
  int m1 = decode(min_cand(3, 0));
  for (int w = tid; w < W; w += kCoopT) s_med[w] = gword(m1, w);
  __syncthreads();
  // ---- m2: farthest from m1, as a minimum of (2Lk - d, position)
  {
    unsigned long long best = ~0ull;
#pragma unroll
    for (int j = 0; j < PPT; ++j) {
      if (!own[j] || pos[j] == m1) continue;
      int d = 0;
      for (int w = 0; w < W; ++w) d += __popcll(word(j, w) ^ s_med[w]);
      const unsigned long long key = ((unsigned long long)(a.twoLk - d) << 24) | (unsigned long long)pos[j];
      best = key < best ? key : best;
    }
    put_cand(3, 1, block_min_u64(best));
  }
  grid_sync(a.bar, nblk, a.err);
  int m2 = decode(min_cand(3, 1));

  int delta[PPT], in1[PPT];
#pragma unroll
  for (int j = 0; j < PPT; ++j) in1[j] = 0;
  int iters = 0, conv = 0, am1 = m1, am2 = m2;
  for (int it = 1; it <= a.max_iters; ++it) {
    int32_t* hc = a.hist + (it & 1) * nbins;       // this round's histogram
    const int cslot = it % 3;
    // A: delta for own positions, block histogram; clear the next round's
    // histogram and candidate slots (last read two barriers ago)
    __syncthreads();                              // s_med of the previous medoids is free
    for (int w = tid; w < W; w += kCoopT) {
      s_med[w] = gword(m1, w);
      s_med[W + w] = gword(m2, w);
    }
    for (int v = tid; v < nbins; v += kCoopT) s_h[v] = 0;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < PPT; ++j) {
      delta[j] = 0;
      if (!own[j]) continue;
      int d = 0;
      for (int w = 0; w < W; ++w) {
        const uint64_t x = word(j, w);
        d += __popcll(x ^ s_med[w]) - __popcll(x ^ s_med[W + w]);
      }
      delta[j] = d;
      atomicAdd(&s_h[d + off], 1);
    }
    {
      int32_t* hn = a.hist + ((it + 1) & 1) * nbins;
      for (int v = blockIdx.x * kCoopT + tid; v < nbins; v += (int)nblk * kCoopT) st_ag(hn + v, 0);
    }
    __syncthreads();
    {
      int32_t* hp = a.hpart + (int64_t)blockIdx.x * nbins;
      for (int v = tid; v < nbins; v += kCoopT) {
        const int h = s_h[v];
        st_ag(hp + v, h);
        if (h) atomicAdd(hc + v, h);
      }
    }
    grid_sync(a.bar, nblk, a.err);
    // B: threshold (every block alike), ties of lower blocks, assignment in
    // position order; batch changes update the batch-1 counts
    for (int v = tid; v < nbins; v += kCoopT) s_h[v] = ld_ag(hc + v);
    if (tid == 0) {                               // defaults that keep indices in range
      s_thr = nbins - 1 - off;
      s_q = n1;
    }
    for (int q = tid; q < LE; q += kCoopT) s_c[q] = 0;
    if (tid == 0) s_tot[0] = 0;
    __syncthreads();
    {
      const int pb = (nbins + kCoopT - 1) / kCoopT;
      const int v0 = min(nbins, tid * pb), v1 = min(nbins, v0 + pb);
      int local = 0;
      for (int v = v0; v < v1; ++v) local += s_h[v];
      int total;
      int cum = block_excl_scan<kCoopT>(local, &total);
      for (int v = v0; v < v1; ++v) {
        const int h = s_h[v];
        if (cum < n1 && cum + h >= n1) {
          s_thr = v - off;
          s_q = n1 - cum;
        }
        cum += h;
      }
    }
    __syncthreads();
    const int thr = s_thr, q = s_q;
    int pre;
    {
      int lower = 0;
      for (int b = tid; b < (int)blockIdx.x; b += kCoopT) lower += ld_ag(a.hpart + (int64_t)b * nbins + thr + off);
      int total;
      block_excl_scan<kCoopT>(lower, &total);
      pre = total;
    }
#pragma unroll
    for (int j = 0; j < PPT; ++j) {
      int ties;
      const int x = block_excl_scan<kCoopT>(own[j] && delta[j] == thr ? 1 : 0, &ties);
      if (own[j]) {
        const int d = delta[j];
        const int nw = d < thr ? 1 : (d > thr ? 0 : (pre + x < q ? 1 : 0));
        if (nw != in1[j]) {
          const int sgn = nw ? 1 : -1;
          for_cols(j, [&](int col, bool ok) { atomicAdd(&s_c[col], ok ? sgn : 0); });
          atomicAdd(&s_tot[0], (unsigned long long)(int64_t)(sgn * ones[j]));
          in1[j] = nw;
        }
      }
      pre += ties;
    }
    __syncthreads();
    for (int qq = tid; qq < LE; qq += kCoopT)
      if (s_c[qq]) atomicAdd(&a.cnt[qq], s_c[qq]);
    if (tid == 0 && s_tot[0]) atomicAdd(&a.tot[0], s_tot[0]);
    am1 = m1;
    am2 = m2;
    iters = it;
    grid_sync(a.bar, nblk, a.err);
    // C: centroid candidates per batch
    for (int qq = tid; qq < LE; qq += kCoopT) {
      const int c1 = ld_ag(a.cnt + qq);
      s_c[qq] = c1;
      s_c[LE + qq] = s_all[qq] - c1;
    }
    if (tid == 0) {
      const unsigned long long t1s = ld_ag64(a.tot);
      s_tot[0] = t1s;
      s_tot[1] = tot_all - t1s;
    }
    __syncthreads();
    {
      unsigned long long b0 = ~0ull, b1 = ~0ull;
#pragma unroll
      for (int j = 0; j < PPT; ++j) {
        if (!own[j]) continue;
        const int c = in1[j] ? 0 : 1;
        const unsigned long long key = dist_key(j, s_c + c * LE, c == 0 ? n1 : N - n1, s_tot[c]);
        if (c == 0) b0 = key < b0 ? key : b0;
        else b1 = key < b1 ? key : b1;
      }
      put_cand(cslot, 0, block_min_u64(b0));
      put_cand(cslot, 1, block_min_u64(b1));
    }
    grid_sync(a.bar, nblk, a.err);
    // D: new centroids; stop when they repeat (same decision in every block)
    const int n1c = decode(min_cand(cslot, 0));
    const int n2c = decode(min_cand(cslot, 1));
    if (n1c == m1 && n2c == m2) {
      conv = 1;
      break;
    }
    m1 = n1c;
    m2 = n2c;
  }
#pragma unroll
  for (int j = 0; j < PPT; ++j)
    if (own[j]) a.in1[a.order[pos[j]]] = in1[j];
  if (blockIdx.x == 0 && tid == 0) {
    a.state[ST_ITERS] = iters;
    a.state[ST_CONV] = conv;
    a.state[ST_AM1] = a.order[am1];
    a.state[ST_AM2] = a.order[am2];
  }
}

// Clears the scratch of one call (a kernel rather than memset nodes, so that
// the sequence can be captured in a graph).
__global__ void __launch_bounds__(kT)
sch_init(int32_t* __restrict__ hist, int nbins2, int32_t* __restrict__ cnt_orig,
         int32_t* __restrict__ cnt, int LE2, unsigned long long* __restrict__ tot,
         unsigned long long* __restrict__ cand, unsigned* __restrict__ bar,
         int32_t* __restrict__ err, int64_t* __restrict__ state) {
  const int g = blockIdx.x * kT + threadIdx.x, stride = gridDim.x * kT;
  for (int q = g; q < nbins2; q += stride) hist[q] = 0;
  for (int q = g; q < LE2; q += stride) {
    cnt_orig[q] = 0;
    cnt[q] = 0;
  }
  if (g < 4) tot[g] = 0;
  if (g < 8) cand[g] = ~0ull;
  if (g < ST_NWORDS) state[g] = 0;
  if (g == 0) {
    *bar = 0;
    *err = 0;
  }
}

// ------------------------------------------------ finish
// Eq. 2 before / after and the guard decision (block 0), and the batch-1
// count of each kSel-token block of token indices. The batch-2 column counts
// are the all-token counts minus the batch-1 counts.
__global__ void __launch_bounds__(kSel)
sch_fin_count(int N, int LE, int keep_if_worse, int trivial, const int32_t* __restrict__ in1,
              const int32_t* __restrict__ cnt, const int32_t* __restrict__ cnt_orig,
              int32_t* __restrict__ blkcnt, int64_t* __restrict__ state) {
  if (blockIdx.x == 0) {
    int a = 0, b = 0;
    for (int q = threadIdx.x; q < LE; q += kSel) {
      const int o0 = cnt_orig[q], o1 = cnt_orig[LE + q];
      a += (o0 > 0) + (o1 > 0);
      if (!trivial) {
        const int c1 = cnt[q];
        b += (c1 > 0) + (o0 + o1 - c1 > 0);
      }
    }
    int before, after;
    block_excl_scan<kSel>(a, &before);
    block_excl_scan<kSel>(b, &after);
    if (trivial) after = before;
    if (threadIdx.x == 0) {
      state[ST_BEFORE] = before;
      state[ST_AFTER] = after;
      state[ST_USE_ORIG] = (trivial || (keep_if_worse && after > before)) ? 1 : 0;
    }
  }
  if (trivial) return;
  const int i = blockIdx.x * kSel + threadIdx.x;
  int tot1;
  block_excl_scan<kSel>((i < N && in1[i] != 0) ? 1 : 0, &tot1);
  if (threadIdx.x == 0) blkcnt[blockIdx.x] = tot1;
}

// perm by stable compaction (batch 1 ascending, then batch 2), demand, info.
__global__ void __launch_bounds__(kSel)
sch_fin_scatter(int N, int n1, int LE, int trivial, const int32_t* __restrict__ in1,
                const int32_t* __restrict__ cnt, const int32_t* __restrict__ cnt_orig,
                const int32_t* __restrict__ blkcnt, const int64_t* __restrict__ state,
                const int32_t* __restrict__ err, int32_t* __restrict__ perm,
                int32_t* __restrict__ demand, int64_t* __restrict__ info,
                int32_t* __restrict__ err_out) {
  const bool use_orig = state[ST_USE_ORIG] != 0;
  const int i = blockIdx.x * kSel + threadIdx.x;
  if (use_orig) {
    if (i < N) perm[i] = i;                       // [0, n1) then [n1, N), each ascending
  } else {
    const int nb = (int)gridDim.x;
    int lower = 0, all = 0;
    for (int b = threadIdx.x; b < nb; b += kSel) {
      const int c = blkcnt[b];
      all += c;
      if (b < (int)blockIdx.x) lower += c;
    }
    int tot1, below;
    block_excl_scan<kSel>(all, &tot1);
    block_excl_scan<kSel>(lower, &below);
    const int one = (i < N && in1[i] != 0) ? 1 : 0;
    int blk;
    const int x = block_excl_scan<kSel>(one, &blk);
    if (i < N) perm[one ? below + x : tot1 + i - (below + x)] = i;
  }
  if (blockIdx.x != 0) return;
  if (demand)
    for (int q = threadIdx.x; q < LE; q += kSel) {
      const int o0 = cnt_orig[q], o1 = cnt_orig[LE + q];
      const int c1 = use_orig ? o0 : cnt[q];
      demand[q] = c1;
      demand[LE + q] = o0 + o1 - c1;
    }
  if (threadIdx.x == 0) {
    // a bounded wait that timed out in the round loop marks the result
    info[0] = (*err) ? -1 : (trivial ? 0 : state[ST_ITERS]);
    if (*err && err_out) *err_out = 1;
    info[1] = trivial ? 1 : state[ST_CONV];
    info[2] = trivial ? -1 : state[ST_AM1];
    info[3] = trivial ? -1 : state[ST_AM2];
    info[4] = state[ST_BEFORE];
    info[5] = use_orig ? state[ST_BEFORE] : state[ST_AFTER];
    info[6] = (!trivial && use_orig) ? 1 : 0;
    info[7] = n1;
  }
}

// ---------------------------------------------------------------- one block
// Up to kSmallN tokens whose packed paths fit in LDS (decode-sized units and
// the small nodes of a B-way split): every step in one block and one launch,
// all state in LDS. Same results as the multi-kernel path, step for step:
// signature order by a bitonic sort under the lowest-differing-bit rule, m1
// and m2, then per round the delta histogram, the threshold with the tie
// quota taken in signature order, the batch-1 column counts, and both
// centroids as (distance sum, signature rank) minima; the guard and outputs.
// Per-token sums are spread over (token, word) items with LDS atomics, so the
// work of a few tokens still runs on all waves of the block; a centroid
// candidate is one 32-bit key (sum << 10 | rank) reduced with DPP moves, and
// the sort's in-wave stages exchange through lane shuffles, not LDS.
constexpr int kSmallN = kSel;
constexpr int kSmallRankBits = 10;               // signature rank < kSmallN
constexpr int kSmallMaxLk = 2048;                // sums < kSmallN * 2 L k fit 22 bits
constexpr int kSmallPre = 8;                     // 16-byte route pieces in flight per thread
constexpr size_t kSmallMaxLds = 140 * 1024;
constexpr int kSmallBatch = 64;                  // nodes per launch (one block each)
static_assert(kSmallN <= (1 << kSmallRankBits), "rank field");
static_assert((int64_t)kSmallN * 2 * kSmallMaxLk <= (1ll << (32 - kSmallRankBits)), "sum field");

// The nodes of one launch: block b splits the n[b] tokens at perm[lo[b] ...]
// with n1[b] in batch 1 and writes info row row[b].
struct SmallNodes {
  int32_t lo[kSmallBatch], n[kSmallBatch], n1[kSmallBatch], row[kSmallBatch];
};

struct SmallLds {
  size_t bits, cnt_all, cnt1, cnt_orig, hist, idx, rank, ones, dbin, in1, sall, s1, skey, stok,
      total;
};

__host__ __device__ inline size_t small_align(size_t v) { return (v + 15) & ~(size_t)15; }

__host__ __device__ inline SmallLds small_lds(int N, int W, int LE, int nbins) {
  int NP = 1;
  while (NP < N) NP <<= 1;
  SmallLds o{};
  size_t p = 0;
  o.bits = p;     p = small_align(p + (size_t)N * W * 8);
  o.cnt_all = p;  p = small_align(p + (size_t)LE * 4);
  o.cnt1 = p;     p = small_align(p + (size_t)LE * 4);
  o.cnt_orig = p; p = small_align(p + (size_t)LE * 4);
  o.hist = p;     p = small_align(p + (size_t)nbins * 4);
  o.idx = p;      p = small_align(p + (size_t)N * 4);
  o.rank = p;     p = small_align(p + (size_t)N * 4);
  o.ones = p;     p = small_align(p + (size_t)N * 4);
  o.dbin = p;     p = small_align(p + (size_t)N * 4);
  o.in1 = p;      p = small_align(p + (size_t)N * 4);
  o.sall = p;     p = small_align(p + (size_t)N * 4);
  o.s1 = p;       p = small_align(p + (size_t)N * 4);
  o.skey = p;     p = small_align(p + (size_t)(NP >= 128 ? NP : 0) * 8);
  o.stok = p;     p = small_align(p + (size_t)(NP >= 128 ? NP : 0) * 4);
  o.total = p;
  return o;
}

// DPP move within rows of 16 lanes (lanes without a source keep `old`)
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t small_dpp(uint32_t old, uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, CTRL, ROWS, 0xf, false);
}

// Minimum over the wave (every lane active), in every lane: row_shr 1, 2, 4, 8
// within rows of 16, then row 15 into rows 1 and 3, row 31 into rows 2 and 3.
__device__ __forceinline__ uint32_t small_wave_min(uint32_t v) {
  v = min(v, small_dpp<0x111, 0xf>(~0u, v));
  v = min(v, small_dpp<0x112, 0xf>(~0u, v));
  v = min(v, small_dpp<0x114, 0xf>(~0u, v));
  v = min(v, small_dpp<0x118, 0xf>(~0u, v));
  v = min(v, small_dpp<0x142, 0xa>(~0u, v));
  v = min(v, small_dpp<0x143, 0xc>(~0u, v));
  return (uint32_t)__builtin_amdgcn_readlane((int)v, kWave - 1);
}

// Inclusive prefix sum over the wave (every lane active), same moves.
__device__ __forceinline__ int small_wave_scan(int v) {
  v += (int)small_dpp<0x111, 0xf>(0u, (uint32_t)v);
  v += (int)small_dpp<0x112, 0xf>(0u, (uint32_t)v);
  v += (int)small_dpp<0x114, 0xf>(0u, (uint32_t)v);
  v += (int)small_dpp<0x118, 0xf>(0u, (uint32_t)v);
  v += (int)small_dpp<0x142, 0xa>(0u, (uint32_t)v);
  v += (int)small_dpp<0x143, 0xc>(0u, (uint32_t)v);
  return v;
}

// Block-wide minima of two keys at once (all kSel threads call it).
__device__ __forceinline__ void small_block_min2(uint32_t& a, uint32_t& b, uint32_t* red) {
  constexpr int NWv = kSel / kWave;
  a = small_wave_min(a);
  b = small_wave_min(b);
  if (lane_id() == 0) {
    red[threadIdx.x / kWave] = a;
    red[NWv + threadIdx.x / kWave] = b;
  }
  __syncthreads();
  uint32_t ra = red[0], rb = red[NWv];
#pragma unroll
  for (int w = 1; w < NWv; ++w) {
    ra = min(ra, red[w]);
    rb = min(rb, red[NWv + w]);
  }
  __syncthreads();
  a = ra;
  b = rb;
}

// Block-wide exclusive scan; the block total goes to *total.
__device__ __forceinline__ int small_block_scan(int v, int* total, int* red) {
  constexpr int NWv = kSel / kWave;
  const int inc = small_wave_scan(v);
  if (lane_id() == kWave - 1) red[threadIdx.x / kWave] = inc;
  __syncthreads();
  const int me = threadIdx.x / kWave;
  int base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NWv; ++w) {
    const int x = red[w];
    base += w < me ? x : 0;
    tot += x;
  }
  __syncthreads();
  *total = tot;
  return base + inc - v;
}

// ids_in == 0: token i of the node is routes row i, and perm[lo + j] receives
// the node-local index of the token at position j of the split (batch 1, then
// batch 2, each ascending). ids_in == 1: token i is routes row perm[lo + i],
// and the same positions receive those row ids (the node's tokens reordered
// in place). demand (single node only) and info may be null.
__global__ void __launch_bounds__(kSel)
sch_small(const uint8_t* __restrict__ routes, const SmallNodes nodes, int ids_in, int L, int E,
          int k, int W, int max_iters, int keep, int nbins, int32_t* __restrict__ perm,
          int32_t* __restrict__ demand, int64_t* __restrict__ info_rows) {
  extern __shared__ __attribute__((aligned(16))) unsigned char s_lds[];
  __shared__ uint32_t s_red[2 * kSel / kWave];
  __shared__ int s_t, s_below;
  const int tid = threadIdx.x;
  const int N = nodes.n[blockIdx.x], n1 = nodes.n1[blockIdx.x], lo = nodes.lo[blockIdx.x];
  int64_t* const info = info_rows ? info_rows + 8 * (int64_t)nodes.row[blockIdx.x] : nullptr;
  if (N == 0) {                                  // an empty node: nothing to split
    if (info && tid < 8) info[tid] = (tid == 1) ? 1 : (tid == 2 || tid == 3) ? -1 : 0;
    return;
  }
  const bool trivial = n1 == 0 || n1 == N;
  const int LE = L * E, Lk = L * k, NW = N * W;
  const SmallLds o = small_lds(N, W, LE, nbins);
  uint64_t* const bits = reinterpret_cast<uint64_t*>(s_lds + o.bits);
  uint32_t* const bits32 = reinterpret_cast<uint32_t*>(s_lds + o.bits);
  int* const cnt_all = reinterpret_cast<int*>(s_lds + o.cnt_all);
  int* const cnt1 = reinterpret_cast<int*>(s_lds + o.cnt1);
  int* const cnt_orig = reinterpret_cast<int*>(s_lds + o.cnt_orig);
  int* const hist = reinterpret_cast<int*>(s_lds + o.hist);
  int* const idx = reinterpret_cast<int*>(s_lds + o.idx);
  int* const rank = reinterpret_cast<int*>(s_lds + o.rank);
  int* const ones = reinterpret_cast<int*>(s_lds + o.ones);
  int* const dbin = reinterpret_cast<int*>(s_lds + o.dbin);
  int* const in1 = reinterpret_cast<int*>(s_lds + o.in1);
  int* const sall = reinterpret_cast<int*>(s_lds + o.sall);
  int* const s1 = reinterpret_cast<int*>(s_lds + o.s1);
  uint64_t* const skey = reinterpret_cast<uint64_t*>(s_lds + o.skey);
  int* const stok = reinterpret_cast<int*>(s_lds + o.stok);
  int* const s_redi = reinterpret_cast<int*>(s_red);
  int* const gid = s1;                           // routes row of each token until the rounds
  const int my_id = tid < N ? (ids_in ? perm[lo + tid] : tid) : -1;
  if (tid < N) gid[tid] = my_id;

  for (int q = tid; q < 2 * NW; q += kSel) bits32[q] = 0;
  for (int c = tid; c < LE; c += kSel) {
    cnt_all[c] = 0;
    cnt_orig[c] = 0;
  }
  for (int i = tid; i < N; i += kSel) {
    ones[i] = 0;
    sall[i] = 0;
    dbin[i] = 0;
  }
  __syncthreads();

  // paths: bit l*E+e of token i for each id e < E of its route; a bit set for
  // the first time counts once towards |r_i| and its column
  int my_ones = 0;
  auto set_bit = [&](int tok, int l, int e) {
    if (e >= E) return;
    const int col = l * E + e;
    const uint32_t m = 1u << (col & 31);
    if (atomicOr(&bits32[tok * 2 * W + (col >> 5)], m) & m) return;
    ++my_ones;
    atomicAdd(&ones[tok], 1);
    atomicAdd(&cnt_all[col], 1);
    if (tok < n1) atomicAdd(&cnt_orig[col], 1);
  };
  // 16-byte pieces when rows allow it: the node's rows back to back (ids_in
  // == 0), or whole rows of 16-byte multiples (ids_in == 1); else bytes
  const int64_t nbytes = (int64_t)N * Lk;
  const bool aligned = (reinterpret_cast<uintptr_t>(routes) & 15) == 0;
  const int64_t npiece = !aligned ? 0 : !ids_in ? nbytes / 16 : (Lk % 16 == 0 ? nbytes / 16 : 0);
  const int ppr = Lk / 16;                       // pieces per row (ids_in, Lk % 16 == 0)
  auto piece_at = [&](int64_t q, int& tok, int& pos) -> const u32x4_t* {
    if (!ids_in) {
      tok = (int)(q * 16 / Lk);
      pos = (int)(q * 16 - (int64_t)tok * Lk);
      return reinterpret_cast<const u32x4_t*>(routes) + q;
    }
    tok = (int)(q / ppr);
    pos = (int)(q - (int64_t)tok * ppr) * 16;
    return reinterpret_cast<const u32x4_t*>(routes + (int64_t)gid[tok] * Lk + pos);
  };
  for (int64_t q0 = 0; q0 < npiece; q0 += (int64_t)kSmallPre * kSel) {
    u32x4_t v[kSmallPre];
#pragma unroll
    for (int u = 0; u < kSmallPre; ++u) {
      const int64_t q = q0 + (int64_t)u * kSel + tid;
      int tok, pos;
      if (q < npiece) v[u] = *piece_at(q, tok, pos);
    }
#pragma unroll
    for (int u = 0; u < kSmallPre; ++u) {
      const int64_t q = q0 + (int64_t)u * kSel + tid;
      if (q < npiece) {
        int tok, pos;
        (void)piece_at(q, tok, pos);
        int l = pos / k, j = pos - l * k;
#pragma unroll
        for (int c = 0; c < 16; ++c) {
          set_bit(tok, l, (int)((v[u][c >> 2] >> (8 * (c & 3))) & 0xff));
          if (++j == k) {
            j = 0;
            if (++l == L) {
              l = 0;
              ++tok;
            }
          }
        }
      }
    }
  }
  for (int64_t q = npiece * 16 + tid; q < nbytes; q += kSel) {
    const int tok = (int)(q / Lk), pos = (int)(q - (int64_t)tok * Lk);
    set_bit(tok, pos / k, routes[(int64_t)gid[tok] * Lk + pos]);
  }
  int tot_all = 0;
  (void)small_block_scan(my_ones, &tot_all, s_redi);  // its barriers publish bits and counts

  // per token: sum over its columns of cnt[]; accumulated into out[] (zeroed)
  auto col_sums = [&](const int* cnt, int* out) {
    for (int q = tid; q < NW; q += kSel) {
      const int lo = (q % W) * 64;
      int sum = 0;
      for (uint64_t x = bits[q]; x; x &= x - 1) sum += cnt[lo + __builtin_ctzll(x)];
      if (sum) atomicAdd(&out[q / W], sum);
    }
  };
  col_sums(cnt_all, sall);

  int iters = 0, converged = 1, med0 = -1, med1 = -1;
  if (trivial) {                                 // one batch empty: the input split stands
    for (int i = tid; i < N; i += kSel) in1[i] = i < n1 ? 1 : 0;
    for (int col = tid; col < LE; col += kSel) cnt1[col] = cnt_orig[col];
    __syncthreads();
  } else {
    // signature order: bitonic sort of (key, token), one element per thread.
    // The key is word 0 bit-reversed and inverted, so ascending keys follow the
    // lowest-differing-bit rule on word 0; equal keys compare the later words
    // the same way, then the index. Padding (token -1) sorts last.
    int NP = 1;
    while (NP < N) NP <<= 1;
    auto before = [&](uint64_t ka, int ta, uint64_t kb, int tb) {
      if (ta < 0) return false;
      if (tb < 0) return true;
      if (ka != kb) return ka < kb;
      for (int w = 1; w < W; ++w) {
        const uint64_t x = bits[ta * W + w] ^ bits[tb * W + w];
        if (x) return (bits[ta * W + w] & lowbit(x)) != 0;
      }
      return ta < tb;
    };
    uint64_t key = ~0ull;
    int tk = -1;
    if (tid < N) {
      key = ~__builtin_bitreverse64(bits[tid * W]);
      tk = tid;
    }
    for (int kk = 2; kk <= NP; kk <<= 1)
      for (int j = kk >> 1; j > 0; j >>= 1) {
        uint64_t pk;
        int pt;
        if (j < kWave) {
          pk = __shfl_xor(key, j, kWave);
          pt = __shfl_xor(tk, j, kWave);
        } else {                                   // NP >= 128 here
          if (tid < NP) {
            skey[tid] = key;
            stok[tid] = tk;
          }
          __syncthreads();
          pk = tid < NP ? skey[tid ^ j] : key;
          pt = tid < NP ? stok[tid ^ j] : tk;
          __syncthreads();
        }
        // the lower position of an ascending pair keeps the element that comes first
        const bool asc = (tid & kk) == 0, low = (tid & j) == 0;
        const bool pfirst = before(pk, pt, key, tk);
        if (asc == low ? pfirst : !pfirst) {
          key = pk;
          tk = pt;
        }
      }
    if (tid < N) {
      idx[tid] = tk;
      rank[tk] = tid;
    }
    __syncthreads();

    // m1: least total distance; m2: farthest from m1 (ties to the lower rank)
    auto pack = [](int64_t v, int r) { return ((uint32_t)v << kSmallRankBits) | (uint32_t)r; };
    uint32_t c1 = ~0u, c2 = ~0u;
    for (int i = tid; i < N; i += kSel)
      c1 = min(c1, pack((int64_t)N * ones[i] + tot_all - 2 * (int64_t)sall[i], rank[i]));
    small_block_min2(c1, c2, s_red);
    int m1 = idx[c1 & (kSmallN - 1)];
    for (int q = tid; q < NW; q += kSel) {
      const int d = __popcll(bits[q] ^ bits[m1 * W + q % W]);
      if (d) atomicAdd(&dbin[q / W], d);
    }
    __syncthreads();
    c1 = ~0u;
    c2 = ~0u;
    for (int i = tid; i < N; i += kSel)
      if (i != m1) c1 = min(c1, pack(2 * Lk - dbin[i], rank[i]));
    small_block_min2(c1, c2, s_red);
    int m2 = idx[c1 & (kSmallN - 1)];

    const int off = 2 * Lk;                        // delta in [-2Lk, 2Lk]
    converged = 0;
    for (int it = 1; it <= max_iters; ++it) {
      iters = it;
      for (int b = tid; b < nbins; b += kSel) hist[b] = 0;
      for (int i = tid; i < N; i += kSel) {
        dbin[i] = off;
        s1[i] = 0;
      }
      for (int col = tid; col < LE; col += kSel) cnt1[col] = 0;
      __syncthreads();
      for (int q = tid; q < NW; q += kSel) {
        const int w = q % W;
        const uint64_t x = bits[q];
        const int d = __popcll(x ^ bits[m1 * W + w]) - __popcll(x ^ bits[m2 * W + w]);
        if (d) atomicAdd(&dbin[q / W], d);
      }
      __syncthreads();
      for (int i = tid; i < N; i += kSel) atomicAdd(&hist[dbin[i]], 1);
      __syncthreads();
      // threshold bin t: fewer than n1 tokens lie below it, at least n1 up to it
      const int per = (nbins + kSel - 1) / kSel;
      const int b0 = min(nbins, tid * per), b1 = min(nbins, b0 + per);
      int mine = 0;
      for (int b = b0; b < b1; ++b) mine += hist[b];
      int total = 0;
      const int below = small_block_scan(mine, &total, s_redi);
      if (below < n1 && below + mine >= n1) {
        int cum = below;
        for (int b = b0; b < b1; ++b) {
          if (cum + hist[b] >= n1) {
            s_t = b;
            s_below = cum;
            break;
          }
          cum += hist[b];
        }
      }
      __syncthreads();
      const int t = s_t, quota = n1 - s_below;
      // ties at t go to batch 1 in signature order, up to the quota
      const int tok = tid < N ? idx[tid] : -1;
      const int tie = tok >= 0 && dbin[tok] == t ? 1 : 0;
      const int tpos = small_block_scan(tie, &total, s_redi);
      if (tok >= 0) in1[tok] = (dbin[tok] < t || (tie && tpos < quota)) ? 1 : 0;
      __syncthreads();
      int my1 = 0;
      for (int q = tid; q < NW; q += kSel)
        if (in1[q / W]) {
          const int lo = (q % W) * 64;
          uint64_t x = bits[q];
          my1 += __popcll(x);
          for (; x; x &= x - 1) atomicAdd(&cnt1[lo + __builtin_ctzll(x)], 1);
        }
      int tot1 = 0;
      (void)small_block_scan(my1, &tot1, s_redi);   // its barriers publish cnt1
      col_sums(cnt1, s1);
      __syncthreads();
      med0 = m1;
      med1 = m2;
      uint32_t a1 = ~0u, a2 = ~0u;
      for (int i = tid; i < N; i += kSel) {
        if (in1[i])
          a1 = min(a1, pack((int64_t)n1 * ones[i] + tot1 - 2 * (int64_t)s1[i], rank[i]));
        else
          a2 = min(a2, pack((int64_t)(N - n1) * ones[i] + (tot_all - tot1) -
                                2 * (int64_t)(sall[i] - s1[i]), rank[i]));
      }
      small_block_min2(a1, a2, s_red);
      const int n1m = idx[a1 & (kSmallN - 1)];
      const int n2m = idx[a2 & (kSmallN - 1)];
      if (n1m == m1 && n2m == m2) {
        converged = 1;
        break;
      }
      m1 = n1m;
      m2 = n2m;
    }
  }

  // Eq. 2 before and after, the guard
  int ob = 0, oa = 0;
  for (int col = tid; col < LE; col += kSel) {
    ob += (cnt_orig[col] > 0) + (cnt_all[col] - cnt_orig[col] > 0);
    oa += (cnt1[col] > 0) + (cnt_all[col] - cnt1[col] > 0);
  }
  int obj_before = 0, obj_after = 0;
  (void)small_block_scan(ob, &obj_before, s_redi);
  (void)small_block_scan(oa, &obj_after, s_redi);
  const bool use_orig = keep && obj_after > obj_before;
  if (use_orig) obj_after = obj_before;

  // perm: batch 1 in ascending index, then batch 2
  const int f = tid < N ? (use_orig ? (tid < n1 ? 1 : 0) : in1[tid]) : 0;
  int nb1 = 0;
  const int pos = small_block_scan(f, &nb1, s_redi);
  if (tid < N) perm[lo + (f ? pos : nb1 + (tid - pos))] = my_id;
  if (demand)
    for (int col = tid; col < LE; col += kSel) {
      const int c = use_orig ? cnt_orig[col] : cnt1[col];
      demand[col] = c;
      demand[LE + col] = cnt_all[col] - c;
    }
  if (info && tid == 0) {
    info[0] = iters;
    info[1] = converged;
    info[2] = med0;
    info[3] = med1;
    info[4] = obj_before;
    info[5] = obj_after;
    info[6] = use_orig ? 1 : 0;
    info[7] = n1;
  }
}

// LDS bytes of the one-block path for a node of n tokens, 0 if it does not
// take that path.
inline size_t small_fit(int64_t n, int L, int E, int k) {
  if (n > kSmallN || (int64_t)L * k >= kSmallMaxLk) return 0;
  const size_t b = small_lds((int)n, (L * E + 63) / 64, L * E, 4 * L * k + 1).total;
  return b <= kSmallMaxLds ? b : 0;
}

// sch_small over the first `count` nodes of the table (lds: the largest
// small_fit among them).
inline hipError_t small_launch(const uint8_t* routes, const SmallNodes& nodes, int count,
                               int ids_in, int L, int E, int k, int max_iters, int keep,
                               size_t lds, int32_t* perm, int32_t* demand, int64_t* info,
                               hipStream_t st) {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&sch_small),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  sch_small<<<dim3(count), dim3(kSel), lds, st>>>(routes, nodes, ids_in, L, E, k,
                                                  (L * E + 63) / 64, max_iters, keep,
                                                  4 * L * k + 1, perm, demand, info);
  return hipGetLastError();
}

struct SchLayout {
  size_t bits, bits_s, key0, key1, key2, skey0, skey1, skey2, sidx, part, ones, ones_s, rank, order, delta,
      in1, cnt, cnt_orig, hist, hpart, tot, state, cand, cand8, blkcnt, bar, total;
};

int rank_groups(int64_t N) {
  return (int)std::min<int64_t>(kMaxRankGroups, ceil_div(N, kChunk));
}

bool coop_shapes(int64_t N, int64_t L, int64_t E, int64_t k) {
  return L * E <= kCoopMaxLE && N < (1 << 24) && 4 * L * k + 1 <= kCoopMaxBins;
}

SchLayout sch_layout(int64_t N, int32_t L, int32_t E, int32_t k) {
  const int64_t W = ((int64_t)L * E + 63) / 64;
  const int64_t LE = (int64_t)L * E;
  const int64_t nbins = 4 * (int64_t)L * k + 1;
  const int64_t nblk = ceil_div(N, kT);
  const int64_t coop_blocks =
      coop_shapes(N, L, E, k) ? std::min<int64_t>(kCoopMaxBlocks, ceil_div(N, kCoopT)) : 0;
  SchLayout s{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + bytes, 256);
    return at;
  };
  s.bits = take(N * W * 8);
  s.bits_s = take(coop_blocks ? N * W * 8 : 0);
  s.key0 = take(N * 8);
  s.key1 = take(N * 8);
  s.key2 = take(N * 8);
  s.skey0 = take(N * 8);
  s.skey1 = take(N * 8);
  s.skey2 = take(N * 8);
  s.sidx = take(N * 4);
  s.part = take((size_t)rank_groups(N) * N * 4);
  s.ones = take(N * 4);
  s.ones_s = take(N * 4);
  s.rank = take(N * 4);
  s.order = take(N * 4);
  s.delta = take(N * 4);
  s.in1 = take(N * 4);
  s.cnt = take(2 * LE * 4);
  s.cnt_orig = take(2 * LE * 4);
  s.hist = take(2 * nbins * 4);
  s.hpart = take(coop_blocks * nbins * 4);
  s.tot = take(4 * 8);
  s.state = take(ST_NWORDS * 8);
  s.cand = take(nblk * 2 * sizeof(Cand));
  s.cand8 = take(8 * 8 * (size_t)std::max<int64_t>(1, coop_blocks));
  s.blkcnt = take(ceil_div(N, kSel) * 4);
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
                            int32_t* perm, int32_t* demand, int64_t* info, int32_t* err_out,
                            void* workspace, size_t ws_bytes, void* stream) {
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
  auto* bits_s = reinterpret_cast<uint64_t*>(ws + lay.bits_s);
  auto* key0 = reinterpret_cast<uint64_t*>(ws + lay.key0);
  auto* key1 = reinterpret_cast<uint64_t*>(ws + lay.key1);
  auto* key2 = reinterpret_cast<uint64_t*>(ws + lay.key2);
  auto* skey0 = reinterpret_cast<uint64_t*>(ws + lay.skey0);
  auto* skey1 = reinterpret_cast<uint64_t*>(ws + lay.skey1);
  auto* skey2 = reinterpret_cast<uint64_t*>(ws + lay.skey2);
  auto* sidx = reinterpret_cast<int32_t*>(ws + lay.sidx);
  auto* part = reinterpret_cast<int32_t*>(ws + lay.part);
  auto* ones = reinterpret_cast<int32_t*>(ws + lay.ones);
  auto* ones_s = reinterpret_cast<int32_t*>(ws + lay.ones_s);
  auto* rank = reinterpret_cast<int32_t*>(ws + lay.rank);
  auto* order = reinterpret_cast<int32_t*>(ws + lay.order);
  auto* delta = reinterpret_cast<int32_t*>(ws + lay.delta);
  auto* in1 = reinterpret_cast<int32_t*>(ws + lay.in1);
  auto* cnt = reinterpret_cast<int32_t*>(ws + lay.cnt);
  auto* cnt_orig = reinterpret_cast<int32_t*>(ws + lay.cnt_orig);
  auto* hist = reinterpret_cast<int32_t*>(ws + lay.hist);
  auto* hpart = reinterpret_cast<int32_t*>(ws + lay.hpart);
  auto* tot = reinterpret_cast<unsigned long long*>(ws + lay.tot);
  auto* state = reinterpret_cast<int64_t*>(ws + lay.state);
  auto* cand = reinterpret_cast<Cand*>(ws + lay.cand);
  auto* cand8 = reinterpret_cast<unsigned long long*>(ws + lay.cand8);
  auto* blkcnt = reinterpret_cast<int32_t*>(ws + lay.blkcnt);
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
  if (const size_t slds = small_fit(N, L, E, k)) {
    SmallNodes one{};
    one.n[0] = (int32_t)N;
    one.n1[0] = (int32_t)n1;
    if (small_launch(routes, one, 1, 0, L, E, k, max_iters, keep_original_if_worse, slds, perm,
                     demand, info, st) == hipSuccess)
      return MOE_OK;
    (void)hipGetLastError();                     // nothing ran: take the general path
  }

  sch_init<<<dim3((unsigned)std::min<int64_t>(64, ceil_div(std::max(2 * nbins, 2 * LE), kT))), blk,
             0, st>>>(hist, 2 * nbins, cnt_orig, cnt, 2 * LE, tot, cand8, bar, err, state);
  MOE_CHECK_LAUNCH();
  if ((int64_t)kPackT * L * k <= kPackMaxBytes)
    sch_pack<true><<<dim3((unsigned)ceil_div(N, kPackT)), dim3(kPackT), 0, st>>>(
        routes, n, L, E, k, W, bits, key0, key1, key2, ones);
  else
    sch_pack<false><<<dim3((unsigned)ceil_div(N, kPackT)), dim3(kPackT), 0, st>>>(
        routes, n, L, E, k, W, bits, key0, key1, key2, ones);
  MOE_CHECK_LAUNCH();

  bool done = false;
  if (!trivial) {
    // signature order: sorted chunks, then every token's rank by lower bounds
    const int nchunks = (int)ceil_div(N, kChunk), ngroups = rank_groups(N);
    sch_sort_chunks<<<dim3(nchunks), dim3(kSortT), 0, st>>>(key0, key1, key2, bits, n, W, skey0,
                                                            skey1, skey2, sidx);
    MOE_CHECK_LAUNCH();
    if (nchunks <= kMergeRankMaxChunks) {
      sch_merge_rank<<<dim3((unsigned)ceil_div(N, kMergeT), ngroups), dim3(kMergeT), 0, st>>>(
          key0, key1, key2, bits, n, W, nchunks, skey0, skey1, skey2, sidx, part);
      MOE_CHECK_LAUNCH();
      sch_rank_sum<<<grid, blk, 0, st>>>(part, ngroups, n, rank, order);
      MOE_CHECK_LAUNCH();
    } else {
      // merge passes, ping-ponging between the sorted keys and the (now
      // unused) unsorted keys with part as the id buffer
      uint64_t *a0 = skey0, *a1 = skey1, *a2 = skey2, *b0 = key0, *b1 = key1, *b2 = key2;
      int32_t *ai = sidx, *bi = part;
      for (int64_t R = kChunk; R < N; R *= 2) {
        const int64_t T = std::min<int64_t>(kMergeTile, 2 * R);
        sch_merge_pass<<<dim3((unsigned)ceil_div(N, T)), dim3(kMergeBT), 0, st>>>(
            a0, a1, a2, ai, bits, n, W, (int)R, b0, b1, b2, bi);
        MOE_CHECK_LAUNCH();
        std::swap(a0, b0);
        std::swap(a1, b1);
        std::swap(a2, b2);
        std::swap(ai, bi);
      }
      sch_rank_sorted<<<grid, blk, 0, st>>>(ai, n, rank, order);
      MOE_CHECK_LAUNCH();
    }
    if (coop_shapes(N, L, E, k)) {
      sch_repack<<<grid, blk, 0, st>>>(bits, ones, order, n, W, bits_s, ones_s);
      MOE_CHECK_LAUNCH();
      const int cus = device_cu_count();
      const int nb = (int)std::max<int64_t>(
          1, std::min<int64_t>({(int64_t)cus, ceil_div(N, kCoopT), (int64_t)kCoopMaxBlocks}));
      const int ppt = (int)ceil_div(ceil_div(N, nb), kCoopT);
      if (ppt <= kCoopMaxPPT) {
        const int ppt_t = ppt <= 1 ? 1 : ppt <= 2 ? 2 : ppt <= 4 ? 4 : ppt <= 8 ? 8 : 16;
        const int Lk = L * k;
        const bool bits_lds = coop_lds(LE, nbins, W, Lk, ppt_t, true, false).total <= kCoopMaxLds;
        const bool rt_lds = E <= 255 &&
            coop_lds(LE, nbins, W, Lk, ppt_t, bits_lds, true).total <= kCoopMaxLds;
        const size_t lds = coop_lds(LE, nbins, W, Lk, ppt_t, bits_lds, rt_lds).total;
        CoopArgs ca{bits_s, ones_s, order, routes, n, W, LE, (int)n1, nbins, off, max_iters,
                    2 * L * k, bits_lds ? 1 : 0, rt_lds ? 1 : 0, E, k, Lk, L, in1, hist, hpart, cnt,
                    cnt_orig, tot, cand8, bar, err, state};
        void* args[] = {&ca};
        const void* fn = ppt_t == 1   ? reinterpret_cast<const void*>(&sch_coop<1>)
                         : ppt_t == 2 ? reinterpret_cast<const void*>(&sch_coop<2>)
                         : ppt_t == 4 ? reinterpret_cast<const void*>(&sch_coop<4>)
                         : ppt_t == 8 ? reinterpret_cast<const void*>(&sch_coop<8>)
                                      : reinterpret_cast<const void*>(&sch_coop<16>);
        // An ordinary launch: nb <= compute units and at least one block fits
        // on a compute unit, so every block becomes resident once the units
        // are free of other work (blocks of kernels on other streams retire
        // without waiting for this one); the barrier waits are bounded in
        // any case. (The cooperative launch API adds nothing to that on this
        // path; processes that used it faulted in the runtime's teardown at
        // exit when traced by the profiler.)
        int per_cu = 0;
        if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) ==
                hipSuccess &&
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kCoopT, lds) ==
                hipSuccess &&
            per_cu >= 1 &&
            hipLaunchKernel(fn, dim3(nb), dim3(kCoopT), args, lds, st) == hipSuccess)
          done = true;
        else
          (void)hipGetLastError();               // nothing ran: take the per-phase path
      }
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
  const dim3 fgrid((unsigned)ceil_div(N, kSel));
  sch_fin_count<<<fgrid, dim3(kSel), 0, st>>>(n, LE, keep_original_if_worse, trivial ? 1 : 0, in1,
                                             cnt, cnt_orig, blkcnt, state);
  MOE_CHECK_LAUNCH();
  sch_fin_scatter<<<fgrid, dim3(kSel), 0, st>>>(n, (int)n1, LE, trivial ? 1 : 0, in1, cnt,
                                               cnt_orig, blkcnt, state, err, perm, demand, info,
                                               err_out);
  MOE_CHECK_LAUNCH();
#undef MOE_TRY
  return MOE_OK;
}

// ==================================================================== B ways
// B-way rebatching by recursive bisection with the two-way scheduler above: a
// node holds n tokens (a range of perm) bound for b batches; b == 1 is a batch,
// otherwise the node's tokens, in their current order, are split with
// n1 = n * (b / 2) / b and the two halves recurse into b / 2 and b - b / 2
// batches. Info rows follow the tree's pre-order; the host walks it level by
// level, and every step on the data is a kernel on the caller's stream.
namespace moe {
namespace {

constexpr int32_t kMaxMultiBatches = 4096;

struct MultiNode {
  int64_t lo, n;
  int32_t b, depth;
};

// Nodes of the recursion in pre-order (sizes depend on N and B only).
std::vector<MultiNode> multi_nodes(int64_t N, int32_t B) {
  std::vector<MultiNode> out, stack{{0, N, B, 0}};
  while (!stack.empty()) {
    const MultiNode v = stack.back();
    stack.pop_back();
    if (v.b == 1) continue;
    out.push_back(v);
    const int32_t bl = v.b / 2;
    const int64_t n1 = v.n * bl / v.b;
    stack.push_back({v.lo + n1, v.n - n1, v.b - bl, v.depth + 1});   // right after left
    stack.push_back({v.lo, n1, bl, v.depth + 1});
  }
  return out;
}

// Batch boundaries on the host (the device kernel below computes the same).
std::vector<int64_t> multi_offsets_host(int64_t N, int32_t B) {
  std::vector<int64_t> off{0};
  std::vector<std::pair<int64_t, int32_t>> stack{{N, B}};
  while (!stack.empty()) {
    const auto v = stack.back();
    stack.pop_back();
    if (v.second == 1) {
      off.push_back(off.back() + v.first);
      continue;
    }
    const int32_t bl = v.second / 2;
    const int64_t n1 = v.first * bl / v.second;
    stack.push_back({v.first - n1, v.second - bl});
    stack.push_back({n1, bl});
  }
  return off;
}

struct MultiLayout {
  size_t sub, routes, tmp, sub_perm, info, total;
};

MultiLayout multi_layout(int64_t N, int32_t L, int32_t E, int32_t k, int32_t B) {
  MultiLayout m{};
  size_t sub = 0;
  for (const MultiNode& v : multi_nodes(N, B))
    if (v.n >= 1) sub = std::max(sub, sch_layout(v.n, L, E, k).total);
  size_t off = align_up(sub, 256);
  m.sub = 0;
  m.routes = off;
  off = align_up(off + (size_t)N * L * k, 256);
  m.tmp = off;
  off = align_up(off + (size_t)N * 4, 256);
  m.sub_perm = off;
  off = align_up(off + (size_t)N * 4, 256);
  m.info = off;                               // one info row when the caller passes none
  off = align_up(off + 8 * sizeof(int64_t), 256);
  m.total = off;
  return m;
}

__global__ void sch_multi_iota(int64_t N, int32_t* __restrict__ ids) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i < N) ids[i] = (int32_t)i;
}

// out[i, :] = routes[ids[i], :] for the n tokens of one node (row = L*k bytes)
__global__ void sch_multi_gather(const uint8_t* __restrict__ routes, const int32_t* __restrict__ ids,
                                 int64_t n, int64_t row, uint8_t* __restrict__ out) {
  const int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (q >= n * row) return;
  const int64_t i = q / row, c = q - i * row;
  out[q] = routes[(int64_t)ids[i] * row + c];
}

// tmp[i] = ids[sub_perm[i]]: the node's tokens in the order its split left them
__global__ void sch_multi_compose(const int32_t* __restrict__ ids, const int32_t* __restrict__ sub_perm,
                                  int64_t n, int32_t* __restrict__ tmp) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i < n) tmp[i] = ids[sub_perm[i]];
}

__global__ void sch_multi_copy(const int32_t* __restrict__ src, int64_t n, int32_t* __restrict__ dst) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i < n) dst[i] = src[i];
}

// The info row of a split of an empty node: nothing to split.
__global__ void sch_multi_info_empty(int64_t* __restrict__ info) {
  const int q = threadIdx.x;
  if (q < 8) info[q] = (q == 1) ? 1 : (q == 2 || q == 3) ? -1 : 0;
}

// offsets[j] for j = 0..B: descend the recursion to batch j's left edge.
__global__ void sch_multi_offsets(int64_t N, int32_t B, int32_t* __restrict__ offsets) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j > B) return;
  if (j == B) {
    offsets[B] = (int32_t)N;
    return;
  }
  int64_t lo = 0, n = N;
  int32_t b = B, jj = j;
  while (b > 1) {
    const int32_t bl = b / 2;
    const int64_t n1 = n * bl / b;
    if (jj < bl) {
      n = n1;
      b = bl;
    } else {
      lo += n1;
      n -= n1;
      jj -= bl;
      b -= bl;
    }
  }
  offsets[j] = (int32_t)lo;
}

__global__ void sch_multi_zero(int64_t n, int32_t* __restrict__ p) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

// demand[b, l, e] = tokens of batch b whose route uses (l, e). Block (c, b)
// counts kDemandChunk tokens of batch b into an LDS histogram when L*E fits
// (else straight into memory), then adds it to demand (zeroed first): many
// blocks per batch keep the LDS atomics on the few (l, e) cells of small E
// from serialising. A token repeating an expert within a layer counts once.
constexpr int kDemandLdsWords = 16384;
constexpr int kDemandChunk = 256;
template <bool LDS>
__global__ void __launch_bounds__(256)
sch_multi_demand(const uint8_t* __restrict__ routes, const int32_t* __restrict__ perm,
                 const int32_t* __restrict__ offsets, int32_t L, int32_t E, int32_t k,
                 int32_t* __restrict__ demand) {
  __shared__ int32_t h[LDS ? kDemandLdsWords : 1];
  const int b = blockIdx.y;
  const int64_t LE = (int64_t)L * E;
  int32_t* const out = demand + (int64_t)b * LE;
  const int64_t lo = offsets[b] + (int64_t)blockIdx.x * kDemandChunk;
  const int64_t hi = min((int64_t)offsets[b + 1], lo + kDemandChunk);
  if (lo >= hi) return;                                // uniform over the block
  if (LDS) {
    for (int64_t q = threadIdx.x; q < LE; q += blockDim.x) h[q] = 0;
    __syncthreads();
  }
  const int64_t total = (hi - lo) * L;
  for (int64_t q = threadIdx.x; q < total; q += blockDim.x) {
    const int64_t p = lo + q % (hi - lo);              // neighbouring threads: neighbouring tokens
    const int l = (int)(q / (hi - lo));
    const uint8_t* r = routes + ((int64_t)perm[p] * L + l) * k;
    for (int j = 0; j < k; ++j) {
      bool seen = false;
      for (int jj = 0; jj < j; ++jj) seen |= r[jj] == r[j];
      if (seen || r[j] >= E) continue;
      const int64_t cell = (int64_t)l * E + r[j];
      if (LDS) atomicAdd(&h[cell], 1);
      else atomicAdd(&out[cell], 1);
    }
  }
  if (LDS) {
    __syncthreads();
    for (int64_t q = threadIdx.x; q < LE; q += blockDim.x)
      if (h[q]) atomicAdd(&out[q], h[q]);
  }
}

}  // namespace
}  // namespace moe

extern "C" size_t moe_schedule_multi_workspace(int64_t N, int32_t L, int32_t E, int32_t k,
                                               int32_t B) {
  if (N < 1 || L < 1 || E < 1 || k < 1 || B < 1 || B > moe::kMaxMultiBatches) return 0;
  return moe::multi_layout(N, L, E, k, B).total;
}

extern "C" int moe_schedule_multi(const uint8_t* routes, int64_t N, int32_t L, int32_t E,
                                  int32_t k, int32_t B, int32_t max_iters,
                                  int32_t keep_original_if_worse, int32_t* perm,
                                  int32_t* batch_offsets, int32_t* demand, int64_t* info,
                                  int32_t* err_out, void* workspace, size_t ws_bytes,
                                  void* stream) {
  using namespace moe;
  MOE_CHECK_ARG(routes && perm && batch_offsets);
  MOE_CHECK_ARG(N >= 1 && L >= 1 && E >= 1 && E <= 256 && k >= 1 && k <= E);
  MOE_CHECK_ARG(B >= 1 && B <= kMaxMultiBatches && max_iters >= 1);
  MOE_CHECK_ARG(keep_original_if_worse == 0 || keep_original_if_worse == 1);
  if (N >= ((int64_t)1 << 26) || (int64_t)L * E >= ((int64_t)1 << 24) ||
      (int64_t)L * k >= ((int64_t)1 << 24))
    return MOE_ERR_UNSUPPORTED;
  const MultiLayout lay = multi_layout(N, L, E, k, B);
  if (!workspace || ws_bytes < lay.total || (reinterpret_cast<uintptr_t>(workspace) & 255))
    return MOE_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace);
  void* sub_ws = ws + lay.sub;
  const size_t sub_bytes = lay.routes;
  auto* rt = reinterpret_cast<uint8_t*>(ws + lay.routes);
  auto* tmp = reinterpret_cast<int32_t*>(ws + lay.tmp);
  auto* sub_perm = reinterpret_cast<int32_t*>(ws + lay.sub_perm);
  auto* info_scratch = reinterpret_cast<int64_t*>(ws + lay.info);
  hipStream_t st = as_stream(stream);
  const int64_t row = (int64_t)L * k;
  if (ceil_div(N * row, 256) > 0x7fffffff) return MOE_ERR_UNSUPPORTED;

  sch_multi_iota<<<dim3((unsigned)ceil_div(N, 256)), dim3(256), 0, st>>>(N, perm);
  MOE_CHECK_LAUNCH();
  // one node through the general two-way path: its routes gathered, split,
  // its range of perm composed with the split's order
  auto multi_split = [&](const MultiNode& v, size_t q) -> int {
    int64_t* const info_row = info ? info + 8 * (int64_t)q : info_scratch;
    int32_t* const ids = perm + v.lo;
    const int64_t n1 = v.n * (v.b / 2) / v.b;
    sch_multi_gather<<<dim3((unsigned)ceil_div(v.n * row, 256)), dim3(256), 0, st>>>(
        routes, ids, v.n, row, rt);
    MOE_CHECK_LAUNCH();
    const int rc = moe_schedule(rt, v.n, L, E, k, n1, max_iters, keep_original_if_worse, sub_perm,
                                nullptr, info_row, err_out, sub_ws, sub_bytes, stream);
    if (rc != MOE_OK) return rc;
    const dim3 g((unsigned)ceil_div(v.n, 256));
    sch_multi_compose<<<g, dim3(256), 0, st>>>(ids, sub_perm, v.n, tmp);
    MOE_CHECK_LAUNCH();
    sch_multi_copy<<<g, dim3(256), 0, st>>>(tmp, v.n, ids);
    MOE_CHECK_LAUNCH();
    return MOE_OK;
  };
  // The nodes of one depth are disjoint ranges of perm, each depending only
  // on its parent: a level's nodes that fit the one-block path run as one
  // launch (a block per node, tokens reordered in place), the others one
  // after another.
  const std::vector<MultiNode> nodes = multi_nodes(N, B);
  int32_t depth_max = 0;
  for (const MultiNode& v : nodes) depth_max = std::max(depth_max, v.depth);
  for (int32_t d = 0; d <= depth_max && !nodes.empty(); ++d) {
    SmallNodes tab{};
    int count = 0;
    size_t lds = 0;
    auto flush = [&]() -> int {
      if (count == 0) return MOE_OK;
      if (small_launch(routes, tab, count, 1, L, E, k, max_iters, keep_original_if_worse, lds,
                       perm, nullptr, info, st) != hipSuccess)
        return MOE_ERR_HIP;
      count = 0;
      lds = 0;
      return MOE_OK;
    };
    for (size_t q = 0; q < nodes.size(); ++q) {
      const MultiNode& v = nodes[q];
      if (v.depth != d) continue;
      if (const size_t b = small_fit(v.n, L, E, k)) {
        tab.lo[count] = (int32_t)v.lo;
        tab.n[count] = (int32_t)v.n;
        tab.n1[count] = (int32_t)(v.n * (v.b / 2) / v.b);
        tab.row[count] = (int32_t)q;
        lds = std::max(lds, b);
        if (++count == kSmallBatch) {
          const int rc = flush();
          if (rc != MOE_OK) return rc;
        }
        continue;
      }
      if (v.n == 0) {                            // an empty node: its info row only
        if (info) {
          sch_multi_info_empty<<<dim3(1), dim3(64), 0, st>>>(info + 8 * (int64_t)q);
          MOE_CHECK_LAUNCH();
        }
        continue;
      }
      const int rc = multi_split(v, q);
      if (rc != MOE_OK) return rc;
    }
    const int rc = flush();
    if (rc != MOE_OK) return rc;
  }
  sch_multi_offsets<<<dim3((unsigned)ceil_div(B + 1, 256)), dim3(256), 0, st>>>(N, B,
                                                                              batch_offsets);
  MOE_CHECK_LAUNCH();
  if (demand) {
    const int64_t LE = (int64_t)L * E;
    const int64_t cells = (int64_t)B * LE;
    if (ceil_div(cells, 256) > 0x7fffffff) return MOE_ERR_UNSUPPORTED;
    sch_multi_zero<<<dim3((unsigned)ceil_div(cells, 256)), dim3(256), 0, st>>>(cells, demand);
    MOE_CHECK_LAUNCH();
    // chunks of the largest batch (sizes depend on N and B only)
    const std::vector<int64_t> off = multi_offsets_host(N, B);
    int64_t largest = 0;
    for (int32_t j = 0; j < B; ++j) largest = std::max(largest, off[j + 1] - off[j]);
    const dim3 g((unsigned)std::max<int64_t>(1, ceil_div(largest, kDemandChunk)), (unsigned)B);
    if (LE <= kDemandLdsWords)
      sch_multi_demand<true><<<g, dim3(256), 0, st>>>(routes, perm, batch_offsets, L, E, k,
                                                       demand);
    else
      sch_multi_demand<false><<<g, dim3(256), 0, st>>>(routes, perm, batch_offsets, L, E, k,
                                                        demand);
    MOE_CHECK_LAUNCH();
  }
  return MOE_OK;
}
