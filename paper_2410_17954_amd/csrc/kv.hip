// KV-cache Merge and Reindex (Sec. 3.3.3). After rebatching, the KV state of
// every token must be found in its new batch: Merge aggregates the original
// batches' caches in global token order (batch 0's tokens, then batch 1's, ...);
// Reindex places global token perm[p] at new position p and tells every global
// token its new batch and position. moe_kv_gather does the row movement of
// both (a copy, bound by HBM), moe_kv_reindex the index maps.
#include "moeflow.h"
#include "common.h"

#include <algorithm>
#include <type_traits>

namespace moe {
namespace {

constexpr int kMaxKvSources = 16;
constexpr int kKvThreads = 256;

struct KvSources {
  const char* base[kMaxKvSources];
  int64_t start[kMaxKvSources + 1];   // global token index of each source's first token
  int n;
};

// dst[l][p] = merged[l][index ? index[p] : p], merged = the sources in global
// order; each source is laid out [L][T_b][row]. A row is copied by tpr threads
// (a power of two) in elements of ELT bytes, 256 / tpr rows per block step.
template <int ELT>
__global__ void __launch_bounds__(kKvThreads)
kv_gather_kernel(KvSources src, int64_t L, int64_t n_out, int64_t row_elts,
                 const int32_t* __restrict__ index, int tpr_shift, char* __restrict__ dst,
                 int32_t* __restrict__ err) {
  using V = typename std::conditional<ELT == 16, uint4, uint8_t>::type;
  const int tpr = 1 << tpr_shift;
  const int sub = threadIdx.x >> tpr_shift;          // row slot within the block
  const int lane = threadIdx.x & (tpr - 1);
  const int rows_per_step = kKvThreads >> tpr_shift;
  const int64_t total = L * n_out;
  const int64_t row_bytes = row_elts * ELT;
  for (int64_t r = (int64_t)blockIdx.x * rows_per_step + sub; r < total;
       r += (int64_t)gridDim.x * rows_per_step) {
    const int64_t l = r / n_out, p = r - l * n_out;
    const int64_t g = index ? (int64_t)index[p] : p;
    int b = 0;
    while (b + 1 < src.n && src.start[b + 1] <= g) ++b;
    if (g < 0 || g >= src.start[src.n]) {           // out-of-range token id: flag, copy nothing
      if (lane == 0) atomicExch(err, 1);
      continue;
    }
    const int64_t tb = src.start[b + 1] - src.start[b];
    const V* s = reinterpret_cast<const V*>(src.base[b] + (l * tb + (g - src.start[b])) * row_bytes);
    V* d = reinterpret_cast<V*>(dst + r * row_bytes);
    for (int64_t c = lane; c < row_elts; c += tpr) d[c] = s[c];
  }
}

// For new position p in batch b: batch_of[perm[p]] = b, pos_of[perm[p]] = p - offsets[b].
__global__ void kv_reindex_kernel(const int32_t* __restrict__ perm, int64_t N,
                                  const int32_t* __restrict__ offsets, int32_t B,
                                  int32_t* __restrict__ batch_of, int32_t* __restrict__ pos_of,
                                  int32_t* __restrict__ err) {
  const int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (p >= N) return;
  int lo = 0, hi = B;                                 // last b with offsets[b] <= p
  while (hi - lo > 1) {
    const int mid = (lo + hi) / 2;
    if (offsets[mid] <= p) lo = mid;
    else hi = mid;
  }
  const int32_t g = perm[p];
  if (g < 0 || g >= N) {
    atomicExch(err, 1);
    return;
  }
  if (batch_of) batch_of[g] = lo;
  if (pos_of) pos_of[g] = (int32_t)(p - offsets[lo]);
}

}  // namespace
}  // namespace moe

extern "C" int moe_kv_gather(const void* const* sources, const int64_t* source_tokens,
                             int32_t n_sources, int64_t L, int64_t row_bytes,
                             const int32_t* index, int64_t n_out, void* dst, int32_t* err,
                             void* stream) {
  using namespace moe;
  MOE_CHECK_ARG(sources && source_tokens && dst && err);
  MOE_CHECK_ARG(n_sources >= 1 && n_sources <= kMaxKvSources && L >= 1 && row_bytes >= 1 &&
                n_out >= 0);
  KvSources src{};
  src.n = n_sources;
  src.start[0] = 0;
  bool aligned = row_bytes % 16 == 0 && (reinterpret_cast<uintptr_t>(dst) & 15) == 0;
  for (int b = 0; b < n_sources; ++b) {
    MOE_CHECK_ARG(source_tokens[b] >= 0 && (source_tokens[b] == 0 || sources[b]));
    src.base[b] = static_cast<const char*>(sources[b]);
    src.start[b + 1] = src.start[b] + source_tokens[b];
    aligned = aligned && (reinterpret_cast<uintptr_t>(sources[b]) & 15) == 0;
  }
  MOE_CHECK_ARG(index || n_out == src.start[n_sources]);   // without index: the merge
  if (n_out == 0) return MOE_OK;
  hipStream_t st = as_stream(stream);
  const int64_t elt = aligned ? 16 : 1;
  const int64_t row_elts = row_bytes / elt;
  int shift = 0;                                     // threads per row: a power of two <= 256
  while (shift < 8 && ((int64_t)2 << shift) <= row_elts) ++shift;
  const int64_t rows = L * n_out;
  const int64_t rows_per_step = kKvThreads >> shift;
  const int64_t want = ceil_div(rows, rows_per_step);
  const unsigned grid = (unsigned)std::min<int64_t>(want, 64 * (int64_t)device_cu_count());
  if (aligned)
    kv_gather_kernel<16><<<dim3(grid), dim3(kKvThreads), 0, st>>>(
        src, L, n_out, row_elts, index, shift, static_cast<char*>(dst), err);
  else
    kv_gather_kernel<1><<<dim3(grid), dim3(kKvThreads), 0, st>>>(
        src, L, n_out, row_elts, index, shift, static_cast<char*>(dst), err);
  MOE_CHECK_LAUNCH();
  return MOE_OK;
}

extern "C" int moe_kv_reindex(const int32_t* perm, int64_t N, const int32_t* batch_offsets,
                              int32_t B, int32_t* batch_of, int32_t* pos_of, int32_t* err,
                              void* stream) {
  using namespace moe;
  MOE_CHECK_ARG(perm && batch_offsets && err && (batch_of || pos_of));
  MOE_CHECK_ARG(N >= 1 && N < ((int64_t)1 << 31) && B >= 1);
  hipStream_t st = as_stream(stream);
  kv_reindex_kernel<<<dim3((unsigned)ceil_div(N, 256)), dim3(256), 0, st>>>(
      perm, N, batch_offsets, B, batch_of, pos_of, err);
  MOE_CHECK_LAUNCH();
  return MOE_OK;
}
