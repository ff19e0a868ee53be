// Forward pass of the routing path predictor (Sec. 3.2): a T5-style
// encoder-decoder whose L heads give every token logits over the E experts of
// each MoE layer, and their sigmoids as activation probabilities (B, S, L, E).
// Everything is float32: on gfx950 the float32 matrix and vector peaks are the
// same, so the contractions (hidden size 32) run as LDS-tiled vector GEMMs.
#include "moeflow.h"
#include "common.h"

#include <algorithm>
#include <vector>

namespace moe {
namespace {

constexpr int kMaxThr = 32;

// Relative-position buckets of one stack (T5): distance n = query - key.
struct RelBuckets {
  int bidirectional;
  int side;        // buckets per sign (num_buckets, or half of it when bidirectional)
  int m;           // exact buckets: distances 0 .. m-1
  int D;           // max_distance: n >= D falls in the last bucket
  int nthr;        // bucket of m <= n < D is m + (number of thr[] <= n)
  int thr[kMaxThr];
};

__device__ __forceinline__ int rel_bucket(const RelBuckets& rb, int n) {
  int ret = 0;
  if (rb.bidirectional) {
    if (n < 0) {
      ret = rb.side;
      n = -n;
    }
  } else if (n < 0) {
    n = 0;
  }
  if (n < rb.m) return ret + n;
  if (n >= rb.D) return ret + rb.side - 1;
  int j = 0;
  for (int q = 0; q < rb.nthr; ++q) j += rb.thr[q] <= n;
  return ret + min(rb.m + j, rb.side - 1);
}

// floor(log2(x)) of a positive 128-bit integer
int ilog2_u128(unsigned __int128 x) {
  int r = -1;
  while (x) {
    x >>= 1;
    ++r;
  }
  return r;
}

// Host: the exact logarithmic buckets. With m and D powers of two the bucket
// of m <= n < D is m + floor((floor(log2(n^a)) - a*log2(m)) / c), a = side - m,
// c = log2(D/m); thr[j-1] = the smallest n with bucket >= m + j.
bool make_buckets(bool bidirectional, int num_buckets, int max_distance, RelBuckets* rb) {
  rb->bidirectional = bidirectional ? 1 : 0;
  rb->side = bidirectional ? num_buckets / 2 : num_buckets;
  rb->m = rb->side / 2;
  rb->D = max_distance;
  const int m = rb->m, a = rb->side - m;
  auto pow2 = [](int v) { return v > 0 && (v & (v - 1)) == 0; };
  if (m < 1 || !pow2(m) || !pow2(max_distance) || max_distance <= m || a > 16) return false;
  const int lm = ilog2_u128(m), c = ilog2_u128((unsigned __int128)(max_distance / m));
  rb->nthr = 0;
  int prev = m;
  for (int n = m; n < max_distance; ++n) {
    unsigned __int128 p = 1;
    for (int q = 0; q < a; ++q) p *= (unsigned __int128)n;   // n < D <= 2^7 keeps n^16 < 2^112
    const int b = std::min(m + (ilog2_u128(p) - a * lm) / c, rb->side - 1);
    while (prev < b) {
      if (rb->nthr >= kMaxThr) return false;
      rb->thr[rb->nthr++] = n;
      ++prev;
    }
  }
  return true;
}

__global__ void rpp_embed(const int32_t* __restrict__ ids, int64_t M, int V, int d,
                          const float* __restrict__ emb, float* __restrict__ x,
                          int32_t* __restrict__ err) {
  const int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (q >= M * d) return;
  const int64_t t = q / d;
  const int c = (int)(q - t * d);
  const int id = ids[t];
  if (id < 0 || id >= V) {
    if (c == 0) atomicExch(err, 1);
    x[q] = 0.f;
    return;
  }
  x[q] = emb[(int64_t)id * d + c];
}

// out = x / sqrt(mean(x^2) + eps) * w; 32 lanes per row (lane c takes columns
// c, c + 32, ...), the sum of squares reduced across them in a fixed order.
__global__ void __launch_bounds__(256)
rpp_rmsnorm(const float* __restrict__ x, int64_t M, int d, const float* __restrict__ w,
            float eps, float* __restrict__ out) {
  const int64_t t = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 5;
  const int lane = threadIdx.x & 31;
  const bool live = t < M;
  const float* r = x + (live ? t : 0) * d;
  float ss = 0.f;
  if (live)
    for (int c = lane; c < d; c += 32) ss += r[c] * r[c];
  for (int o = 16; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 32);
  if (!live) return;
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  for (int c = lane; c < d; c += 32) out[t * d + c] = r[c] * inv * w[c];
}

enum GemmMode { G_STORE = 0, G_ADD = 1, G_RELU = 2, G_SIGMOID = 3 };

// C[M, N] (op)= A[M, K] . W[N, K]^T. 256 threads as 16 x 16, each TM x TN
// outputs (rows ty + 16 i, columns tx + 16 j); K in steps of 16 through LDS.
// G_SIGMOID stores the logits to C and their sigmoids to P.
template <int TM, int TN, int MODE>
__global__ void __launch_bounds__(256)
rpp_gemm(const float* __restrict__ A, int64_t lda, const float* __restrict__ W, int64_t M,
         int64_t N, int64_t K, float* __restrict__ C, int64_t ldc, float* __restrict__ P) {
  constexpr int BM = 16 * TM, BN = 16 * TN, BK = 16;
  __shared__ float As[BK][BM + 1];
  __shared__ float Ws[BK][BN + 1];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int64_t m0 = (int64_t)blockIdx.y * BM, n0 = (int64_t)blockIdx.x * BN;
  float acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = 0.f;
  for (int64_t k0 = 0; k0 < K; k0 += BK) {
    for (int q = threadIdx.x; q < BM * BK; q += 256) {
      const int r = q / BK, c = q % BK;
      const int64_t gr = m0 + r, gc = k0 + c;
      As[c][r] = (gr < M && gc < K) ? A[gr * lda + gc] : 0.f;
    }
    for (int q = threadIdx.x; q < BN * BK; q += 256) {
      const int r = q / BK, c = q % BK;
      const int64_t gr = n0 + r, gc = k0 + c;
      Ws[c][r] = (gr < N && gc < K) ? W[gr * K + gc] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float a[TM], b[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) a[i] = As[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < TN; ++j) b[j] = Ws[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int64_t r = m0 + ty + 16 * i;
    if (r >= M) continue;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int64_t c = n0 + tx + 16 * j;
      if (c >= N) continue;
      float v = acc[i][j];
      if (MODE == G_ADD) v += C[r * ldc + c];
      if (MODE == G_RELU) v = fmaxf(v, 0.f);
      C[r * ldc + c] = v;
      if (MODE == G_SIGMOID) P[r * ldc + c] = 1.0f / (1.0f + __expf(-v));
    }
  }
}

// Attention of (sequence b, head h) for 64 queries per block: softmax over
// keys j of q_i . k_j (+ the bias of distance i - j) with j <= i when causal,
// then the weighted sum of v_j. Keys, values and the head's bias per distance
// (2S - 1 values) are staged in LDS; each query's keys are split over kSplit
// neighbouring lanes (key j goes to lane j mod kSplit), whose running softmax
// states are merged with lane shuffles in a fixed order.
constexpr int kAttQ = 64, kSplit = 4;
template <int DK>
__global__ void __launch_bounds__(kAttQ * kSplit)
rpp_attention(const float* __restrict__ Q, int64_t ldq, const float* __restrict__ Kp,
              const float* __restrict__ Vp, int64_t ldkv, int S, int h_count,
              const float* __restrict__ rel, RelBuckets rb, int use_bias, int causal,
              float* __restrict__ O, int64_t ldo) {
  extern __shared__ float kv_lds[];
  float* const ks = kv_lds;
  float* const vs = kv_lds + (size_t)S * DK;
  float* const bt = vs + (size_t)S * DK;              // bias of distance n at bt[n + S - 1]
  const int h = blockIdx.y, b = blockIdx.z;
  const int64_t base = (int64_t)b * S;
  for (int q = threadIdx.x; q < S * DK; q += blockDim.x) {
    const int j = q / DK, c = q % DK;
    ks[q] = Kp[(base + j) * ldkv + h * DK + c];
    vs[q] = Vp[(base + j) * ldkv + h * DK + c];
  }
  if (use_bias)
    for (int q = threadIdx.x; q < 2 * S - 1; q += blockDim.x)
      bt[q] = rel[rel_bucket(rb, q - (S - 1)) * h_count + h];
  __syncthreads();
  const int split = threadIdx.x % kSplit;
  const int i = blockIdx.x * kAttQ + threadIdx.x / kSplit;
  const bool live = i < S;
  float qv[DK], acc[DK];
#pragma unroll
  for (int c = 0; c < DK; ++c) {
    qv[c] = live ? Q[(base + i) * ldq + h * DK + c] : 0.f;
    acc[c] = 0.f;
  }
  float mx = -INFINITY, den = 0.f;
  const int jend = !live ? 0 : (causal ? i + 1 : S);
  for (int j = split; j < jend; j += kSplit) {
    float sc = 0.f;
#pragma unroll
    for (int c = 0; c < DK; ++c) sc = fmaf(qv[c], ks[j * DK + c], sc);
    if (use_bias) sc += bt[i - j + S - 1];
    const float nm = fmaxf(mx, sc);
    const float scale = __expf(mx - nm), p = __expf(sc - nm);
    den = den * scale + p;
#pragma unroll
    for (int c = 0; c < DK; ++c) acc[c] = fmaf(p, vs[j * DK + c], acc[c] * scale);
    mx = nm;
  }
  // merge the kSplit states of a query (lanes 4q .. 4q+3): pairs at distance 1, then 2
#pragma unroll
  for (int o = 1; o < kSplit; o <<= 1) {
    const float m2 = __shfl_xor(mx, o), d2 = __shfl_xor(den, o);
    const float nm = fmaxf(mx, m2);
    const float s1 = mx == -INFINITY ? 0.f : __expf(mx - nm);
    const float s2 = m2 == -INFINITY ? 0.f : __expf(m2 - nm);
    den = den * s1 + d2 * s2;
#pragma unroll
    for (int c = 0; c < DK; ++c) {
      const float a2 = __shfl_xor(acc[c], o);
      acc[c] = acc[c] * s1 + a2 * s2;
    }
    mx = nm;
  }
  if (!live || split != 0) return;
  const float inv = 1.0f / den;
#pragma unroll
  for (int c = 0; c < DK; ++c) O[(base + i) * ldo + h * DK + c] = acc[c] * inv;
}

constexpr int kMlpRows = 32, kMlpChunk = 64, kMlpSplit = 8;   // fused feed-forward tiles

struct RppOffsets {
  size_t emb, enc_rel, enc_ln, dec_rel, dec_ln, heads, total;
  std::vector<size_t> enc, dec;      // first value of each layer
};

size_t enc_layer_size(const moe_rpp_dims& g) {
  const size_t d = g.d_model, f = g.d_ff;
  return 2 * d + 4 * d * d + 2 * d * f;
}
size_t dec_layer_size(const moe_rpp_dims& g) {
  const size_t d = g.d_model, f = g.d_ff;
  return 3 * d + 8 * d * d + 2 * d * f;
}

RppOffsets rpp_offsets(const moe_rpp_dims& g) {
  RppOffsets o{};
  const size_t d = g.d_model;
  size_t p = 0;
  o.emb = p;
  p += (size_t)g.vocab * d;
  o.enc_rel = p;
  p += (size_t)g.num_buckets * g.n_heads;
  for (int l = 0; l < g.n_enc; ++l) {
    o.enc.push_back(p);
    p += enc_layer_size(g);
  }
  o.enc_ln = p;
  p += d;
  o.dec_rel = p;
  p += (size_t)g.num_buckets * g.n_heads;
  for (int l = 0; l < g.n_dec; ++l) {
    o.dec.push_back(p);
    p += dec_layer_size(g);
  }
  o.dec_ln = p;
  p += d;
  o.heads = p;
  p += (size_t)g.L * g.E * d;
  o.total = p;
  return o;
}

struct RppWs {
  size_t x, y, n, enc, o, qkv, kv, hid, logits, total;
};

RppWs rpp_ws(int64_t M, const moe_rpp_dims& g) {
  RppWs w{};
  size_t off = 0;
  auto take = [&](size_t floats) {
    const size_t at = off;
    off = align_up(off + floats * 4, 256);
    return at;
  };
  const size_t d = g.d_model;
  w.x = take(M * d);
  w.y = take(M * d);
  w.n = take(M * d);
  w.enc = take(M * d);
  w.o = take(M * d);
  w.qkv = take(M * 3 * d);
  w.kv = take(M * 2 * d);
  w.hid = take(M * (size_t)std::max(g.d_ff, kMlpSplit * g.d_model));
  w.logits = take(M * (size_t)g.L * g.E);
  w.total = off;
  return w;
}

bool dims_ok(const moe_rpp_dims* g) {
  if (!g) return false;
  return g->vocab >= 1 && g->d_model >= 1 && g->n_heads >= 1 && g->d_model % g->n_heads == 0 &&
         g->d_ff >= 1 && g->n_enc >= 0 && g->n_dec >= 0 && g->L >= 1 && g->E >= 1 &&
         g->num_buckets >= 2 && g->num_buckets % 2 == 0 && g->max_distance >= 1 && g->eps >= 0.f;
}

template <int MODE>
int gemm(hipStream_t st, const float* A, int64_t lda, const float* W, int64_t M, int64_t N,
         int64_t K, float* C, int64_t ldc, float* P = nullptr) {
  if (N <= 48) {                                  // narrow outputs: 32 x 32 tiles, more blocks
    const dim3 grid((unsigned)ceil_div(N, 32), (unsigned)ceil_div(M, 32));
    rpp_gemm<2, 2, MODE><<<grid, dim3(256), 0, st>>>(A, lda, W, M, N, K, C, ldc, P);
  } else {
    const dim3 grid((unsigned)ceil_div(N, 64), (unsigned)ceil_div(M, 64));
    rpp_gemm<4, 4, MODE><<<grid, dim3(256), 0, st>>>(A, lda, W, M, N, K, C, ldc, P);
  }
  return hipGetLastError() == hipSuccess ? MOE_OK : MOE_ERR_HIP;
}

// Feed-forward block, fused: x[r] += W2 relu(W1 n[r]). Block (row tile, s)
// takes 32 rows through the s-th of kMlpSplit parts of the hidden width, in
// chunks of 64 through LDS (the hidden activations never leave the compute
// unit), loading the next chunk's weights into registers while the current
// one is used, and writes its partial output; rpp_mlp_sum adds the parts and
// the residual in part order. D = d_model (a multiple of 8, <= 64).
template <int D>
__global__ void __launch_bounds__(256)
rpp_mlp(const float* __restrict__ n, int64_t M, const float* __restrict__ W1,
        const float* __restrict__ W2, int dff, float* __restrict__ part) {
  __shared__ float Ns[kMlpRows][D + 1];
  __shared__ float W1s[kMlpChunk][D + 1];             // hidden unit c of the chunk, its D inputs
  __shared__ float Hs[kMlpRows][kMlpChunk + 1];
  __shared__ float W2s[D][kMlpChunk + 1];             // output o, the chunk's hidden units
  constexpr int OPT = D / 8;                          // outputs per thread
  constexpr int PER = kMlpChunk * D / 256;            // weights of each matrix a thread moves
  const int t = threadIdx.x;
  const int64_t r0 = (int64_t)blockIdx.x * kMlpRows;
  const int per_split = (dff + kMlpSplit - 1) / kMlpSplit;
  const int fbeg = min(dff, (int)blockIdx.y * per_split);
  const int fend = min(dff, fbeg + per_split);
  for (int q = t; q < kMlpRows * D; q += 256) {
    const int r = q / D, c = q % D;
    Ns[r][c] = r0 + r < M ? n[(r0 + r) * D + c] : 0.f;
  }
  float w1r[PER], w2r[PER];
  auto fetch = [&](int f0) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int q = t + 256 * u;
      const int c = q / D, k = q % D;                 // W1 row f0 + c, column k
      w1r[u] = f0 + c < fend ? W1[(int64_t)(f0 + c) * D + k] : 0.f;
      const int o = q / kMlpChunk, kk = q % kMlpChunk;   // W2 row o, column f0 + kk
      w2r[u] = f0 + kk < fend ? W2[(int64_t)o * dff + f0 + kk] : 0.f;
    }
  };
  const int r = t >> 3;                               // this thread's row
  const int c0 = (t & 7) * 8;                         // its 8 hidden units of a chunk
  const int o0 = (t & 7) * OPT;                       // its output columns
  float acc[OPT];
#pragma unroll
  for (int j = 0; j < OPT; ++j) acc[j] = 0.f;
  if (fbeg < fend) fetch(fbeg);
  for (int f0 = fbeg; f0 < fend; f0 += kMlpChunk) {
    __syncthreads();                                  // the previous chunk is fully used
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int q = t + 256 * u;
      W1s[q / D][q % D] = w1r[u];
      W2s[q / kMlpChunk][q % kMlpChunk] = w2r[u];
    }
    __syncthreads();
    if (f0 + kMlpChunk < fend) fetch(f0 + kMlpChunk);  // in flight during this chunk
    float hv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) hv[j] = 0.f;
#pragma unroll 8
    for (int k = 0; k < D; ++k) {
      const float a = Ns[r][k];
#pragma unroll
      for (int j = 0; j < 8; ++j) hv[j] = fmaf(a, W1s[c0 + j][k], hv[j]);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) Hs[r][c0 + j] = fmaxf(hv[j], 0.f);
    __syncthreads();
#pragma unroll 8
    for (int k = 0; k < kMlpChunk; ++k) {
      const float a = Hs[r][k];
#pragma unroll
      for (int j = 0; j < OPT; ++j) acc[j] = fmaf(a, W2s[o0 + j][k], acc[j]);
    }
  }
  if (r0 + r < M) {
    float* const out = part + ((int64_t)blockIdx.y * M + r0 + r) * D + o0;
#pragma unroll
    for (int j = 0; j < OPT; ++j) out[j] = acc[j];
  }
}

// x += part[0] + part[1] + ... in part order
__global__ void rpp_mlp_sum(const float* __restrict__ part, int64_t n, float* __restrict__ x) {
  const int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (q >= n) return;
  float v = part[q];
#pragma unroll
  for (int s = 1; s < kMlpSplit; ++s) v += part[s * n + q];
  x[q] += v;
}

int mlp(hipStream_t st, const float* n, int64_t M, int d, const float* W1, const float* W2,
        int dff, float* hid, float* x) {
  // hid (M * dff floats) holds the kMlpSplit partial outputs (M * d each)
  const dim3 grid((unsigned)ceil_div(M, kMlpRows), kMlpSplit);
  switch (d) {
    case 16: rpp_mlp<16><<<grid, dim3(256), 0, st>>>(n, M, W1, W2, dff, hid); break;
    case 32: rpp_mlp<32><<<grid, dim3(256), 0, st>>>(n, M, W1, W2, dff, hid); break;
    case 64: rpp_mlp<64><<<grid, dim3(256), 0, st>>>(n, M, W1, W2, dff, hid); break;
    default: {                                        // other widths: two GEMMs via memory
      int rc = gemm<G_RELU>(st, n, d, W1, M, dff, d, hid, dff);
      if (rc != MOE_OK) return rc;
      return gemm<G_ADD>(st, hid, dff, W2, M, d, dff, x, d);
    }
  }
  if (hipGetLastError() != hipSuccess) return MOE_ERR_HIP;
  rpp_mlp_sum<<<dim3((unsigned)ceil_div(M * d, 256)), dim3(256), 0, st>>>(hid, M * d, x);
  return hipGetLastError() == hipSuccess ? MOE_OK : MOE_ERR_HIP;
}

int attention(hipStream_t st, int dk, const float* Q, int64_t ldq, const float* Kp,
              const float* Vp, int64_t ldkv, int B, int S, int h, const float* rel,
              const RelBuckets& rb, bool use_bias, bool causal, float* O, int64_t ldo) {
  const dim3 grid((unsigned)ceil_div(S, kAttQ), (unsigned)h, (unsigned)B);
  const size_t lds = ((size_t)2 * S * dk + 2 * S) * sizeof(float);
#define MOE_ATT(DKV)                                                                          \
  rpp_attention<DKV><<<grid, dim3(kAttQ * kSplit), lds, st>>>(                               \
      Q, ldq, Kp, Vp, ldkv, S, h, rel, rb, use_bias ? 1 : 0, causal ? 1 : 0, O, ldo)
  switch (dk) {
    case 4: MOE_ATT(4); break;
    case 8: MOE_ATT(8); break;
    case 16: MOE_ATT(16); break;
    case 32: MOE_ATT(32); break;
    case 64: MOE_ATT(64); break;
    default: return MOE_ERR_UNSUPPORTED;
  }
#undef MOE_ATT
  return hipGetLastError() == hipSuccess ? MOE_OK : MOE_ERR_HIP;
}

}  // namespace
}  // namespace moe

extern "C" size_t moe_rpp_weights_count(const moe_rpp_dims* dims) {
  if (!moe::dims_ok(dims)) return 0;
  return moe::rpp_offsets(*dims).total;
}

extern "C" size_t moe_rpp_workspace(int32_t B, int32_t S, const moe_rpp_dims* dims) {
  if (!moe::dims_ok(dims) || B < 1 || S < 1) return 0;
  return moe::rpp_ws((int64_t)B * S, *dims).total;
}

extern "C" int moe_rpp_forward(const int32_t* ids, int32_t B, int32_t S, const moe_rpp_dims* dims,
                               const float* weights, float* probs, float* logits, int32_t* err,
                               void* workspace, size_t ws_bytes, void* stream) {
  using namespace moe;
  MOE_CHECK_ARG(ids && weights && probs && err && dims_ok(dims) && B >= 1 && S >= 1);
  const moe_rpp_dims g = *dims;
  const int d = g.d_model, h = g.n_heads, dk = d / h;
  const int64_t M = (int64_t)B * S;
  if (M * std::max(g.d_ff, 3 * d) >= ((int64_t)1 << 31) / 4 ||
      ((size_t)2 * S * dk + 2 * S) * sizeof(float) > 64 * 1024)
    return MOE_ERR_UNSUPPORTED;
  RelBuckets rb_enc{}, rb_dec{};
  if (!make_buckets(true, g.num_buckets, g.max_distance, &rb_enc) ||
      !make_buckets(false, g.num_buckets, g.max_distance, &rb_dec))
    return MOE_ERR_UNSUPPORTED;
  const RppWs lay = rpp_ws(M, g);
  if (!workspace || ws_bytes < lay.total || (reinterpret_cast<uintptr_t>(workspace) & 255))
    return MOE_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace);
  auto F = [&](size_t off) { return reinterpret_cast<float*>(ws + off); };
  float *x = F(lay.x), *y = F(lay.y), *n = F(lay.n), *enc = F(lay.enc), *o = F(lay.o);
  float *qkv = F(lay.qkv), *kv = F(lay.kv), *hid = F(lay.hid);
  float* lg = logits ? logits : F(lay.logits);
  const RppOffsets wo = rpp_offsets(g);
  const float* W = weights;
  hipStream_t st = as_stream(stream);
  const dim3 rows((unsigned)ceil_div(M * 32, 256));      // 32 lanes per row
  const size_t dd = (size_t)d * d, df = (size_t)d * g.d_ff;
  int rc = MOE_OK;
#define MOE_RC(expr)                  \
  do {                                \
    rc = (expr);                      \
    if (rc != MOE_OK) return rc;      \
  } while (0)

  rpp_embed<<<dim3((unsigned)ceil_div(M * d, 256)), dim3(256), 0, st>>>(ids, M, g.vocab, d,
                                                                      W + wo.emb, x, err);
  MOE_CHECK_LAUNCH();
  for (int l = 0; l < g.n_enc; ++l) {
    const float* p = W + wo.enc[l];
    const float *ln1 = p, *wqkv = p + d, *wout = wqkv + 3 * dd, *ln2 = wout + dd;
    const float *wi = ln2 + d, *wo2 = wi + df;
    rpp_rmsnorm<<<rows, dim3(256), 0, st>>>(x, M, d, ln1, g.eps, n);
    MOE_CHECK_LAUNCH();
    MOE_RC(gemm<G_STORE>(st, n, d, wqkv, M, 3 * d, d, qkv, 3 * d));
    MOE_RC(attention(st, dk, qkv, 3 * d, qkv + d, qkv + 2 * d, 3 * d, B, S, h, W + wo.enc_rel,
                     rb_enc, true, false, o, d));
    MOE_RC(gemm<G_ADD>(st, o, d, wout, M, d, d, x, d));
    rpp_rmsnorm<<<rows, dim3(256), 0, st>>>(x, M, d, ln2, g.eps, n);
    MOE_CHECK_LAUNCH();
    MOE_RC(mlp(st, n, M, d, wi, wo2, g.d_ff, hid, x));
  }
  rpp_rmsnorm<<<rows, dim3(256), 0, st>>>(x, M, d, W + wo.enc_ln, g.eps, enc);
  MOE_CHECK_LAUNCH();
  rpp_embed<<<dim3((unsigned)ceil_div(M * d, 256)), dim3(256), 0, st>>>(ids, M, g.vocab, d,
                                                                      W + wo.emb, y, err);
  MOE_CHECK_LAUNCH();
  for (int l = 0; l < g.n_dec; ++l) {
    const float* p = W + wo.dec[l];
    const float *ln1 = p, *wqkv = p + d, *wout = wqkv + 3 * dd, *ln2 = wout + dd;
    const float *cq = ln2 + d, *ckv = cq + dd, *cout = ckv + 2 * dd, *ln3 = cout + dd;
    const float *wi = ln3 + d, *wo2 = wi + df;
    rpp_rmsnorm<<<rows, dim3(256), 0, st>>>(y, M, d, ln1, g.eps, n);
    MOE_CHECK_LAUNCH();
    MOE_RC(gemm<G_STORE>(st, n, d, wqkv, M, 3 * d, d, qkv, 3 * d));
    MOE_RC(attention(st, dk, qkv, 3 * d, qkv + d, qkv + 2 * d, 3 * d, B, S, h, W + wo.dec_rel,
                     rb_dec, true, true, o, d));
    MOE_RC(gemm<G_ADD>(st, o, d, wout, M, d, d, y, d));
    rpp_rmsnorm<<<rows, dim3(256), 0, st>>>(y, M, d, ln2, g.eps, n);
    MOE_CHECK_LAUNCH();
    MOE_RC(gemm<G_STORE>(st, n, d, cq, M, d, d, qkv, d));
    MOE_RC(gemm<G_STORE>(st, enc, d, ckv, M, 2 * d, d, kv, 2 * d));
    MOE_RC(attention(st, dk, qkv, d, kv, kv + d, 2 * d, B, S, h, nullptr, rb_dec, false, false,
                     o, d));
    MOE_RC(gemm<G_ADD>(st, o, d, cout, M, d, d, y, d));
    rpp_rmsnorm<<<rows, dim3(256), 0, st>>>(y, M, d, ln3, g.eps, n);
    MOE_CHECK_LAUNCH();
    MOE_RC(mlp(st, n, M, d, wi, wo2, g.d_ff, hid, y));
  }
  rpp_rmsnorm<<<rows, dim3(256), 0, st>>>(y, M, d, W + wo.dec_ln, g.eps, n);
  MOE_CHECK_LAUNCH();
  MOE_RC(gemm<G_SIGMOID>(st, n, d, W + wo.heads, M, (int64_t)g.L * g.E, d, lg,
                         (int64_t)g.L * g.E, probs));
#undef MOE_RC
  return MOE_OK;
}
