/*
 * moeflow.h -- C ABI of libmoeflow.so, the MI355X (gfx950) hot path of the
 * MoE layer of ExpertFlow (arXiv 2410.17954) executed over route-grouped
 * token batches:
 *
 *   moe_route       softmax top-k gating                        (Sec. 2.1)
 *   moe_route_binarize  routing paths from predictor scores     (Sec. 3.2)
 *   moe_schedule    balanced rebatching of two adjacent batches
 *                   by predicted routing path                   (Sec. 3.3, Eq. 2)
 *   moe_schedule_multi  the same into B batches by recursive bisection
 *   moe_permute     expert-major grouping of (token, choice) pairs
 *   moe_expert_ffn  grouped SwiGLU experts over the resident
 *                   slots of the expert cache                   (Sec. 2.1, 3.4)
 *   moe_combine     gate-weighted sum of expert outputs         (Sec. 2.1)
 *   moe_kv_gather   KV-cache Merge / Reindex row movement       (Sec. 3.3.3)
 *   moe_kv_reindex  new batch and position of every token       (Sec. 3.3.3)
 *   moe_stack_forward   a batch through L residual MoE layers   (Sec. 2.1)
 *   moe_rpp_forward routing path predictor forward pass         (Sec. 3.2)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory: every array argument is DEVICE memory owned by the caller, row-major
 *   and densely packed. The library never allocates, frees or synchronises;
 *   scratch memory comes from a caller-provided workspace whose size the
 *   matching *_workspace query returns (0 means none is needed). The
 *   workspace must be 256-byte aligned. Its contents on entry do not matter.
 * Ordering: every call only enqueues work on `stream` (a hipStream_t passed as
 *   void*; NULL = the default stream) and returns; outputs are valid once that
 *   work completes. Calls on different streams with disjoint outputs and
 *   workspaces may run concurrently. The library keeps no mutable global
 *   state apart from a per-device cache of the device's compute-unit count.
 * Element types: `dtype` selects MOE_BF16 (bfloat16 bit patterns, uint16) or
 *   MOE_F32 for activations and weights. Logits, biases and gate weights are
 *   always float32; ids and maps are int32.
 * Errors: each call returns MOE_OK or a positive moe_status. Arguments are
 *   validated on the host before anything is enqueued; a failed validation
 *   enqueues nothing and touches no device state. MOE_ERR_HIP reports a
 *   launch failure. Nothing throws across the ABI.
 * Device-side preconditions (ids in range, k distinct experts per route
 *   layer, finite values) cannot be checked without synchronising. The
 *   kernels never read or write outside the arrays described here whatever
 *   those values are, but results are unspecified when they are violated.
 */
#ifndef MOEFLOW_H
#define MOEFLOW_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum moe_status {
  MOE_OK = 0,
  MOE_ERR_ARG = 1,          /* null required pointer, bad size or flag     */
  MOE_ERR_UNSUPPORTED = 2,  /* valid request outside what the kernels do   */
  MOE_ERR_WORKSPACE = 3,    /* workspace missing, too small or misaligned  */
  MOE_ERR_HIP = 4           /* a HIP launch or query failed                */
};

enum moe_dtype { MOE_F32 = 0, MOE_BF16 = 1 };

/* Version of this interface; bumped on any incompatible change. */
#define MOEFLOW_ABI_VERSION 2
int moe_abi_version(void);

/* Static, human-readable name of a status code. */
const char* moe_status_str(int status);

/* ------------------------------------------------------------------------
 * moe_route -- gating (Sec. 2.1: scores softmax(x W_g), the k experts with
 * the highest scores, each weighted by its score).
 *
 *   z[t,e]    = sum_h x[t,h] * w_gate[e,h]  (+ bias)       float32 accumulation
 *   idx[t,:]  = the k largest z[t,:], descending; equal logits go to the lower
 *               expert index; -0.0 == +0.0
 *   w[t,j]    = softmax(z[t,:])[idx[t,j]]               (renormalize = 0)
 *             = the same divided by sum_j of it, i.e. the softmax over the k
 *               selected logits                          (renormalize = 1)
 *
 * x        [T,H] dtype     hidden states                     (x-mode)
 * w_gate   [E,H] dtype     router weight, one row per expert (x-mode)
 * bias     float32, NULL (bias_mode 0), [E] (bias_mode 1) or [T,E] (bias_mode 2)
 * logits   [T,E] float32   x-mode: optional output (NULL = not written);
 *                          logits-in mode: required input
 * topk_idx [T,k] int32     output
 * topk_w   [T,k] float32   output
 * Logits-in mode: x == NULL and w_gate == NULL; then bias must be NULL and
 *   the gate is computed from the given logits (dtype and H are ignored).
 * Limits: T >= 1, 1 <= k <= E <= 256; x-mode bf16 needs H % 8 == 0, f32 needs
 *   H >= 1.
 * ---------------------------------------------------------------------- */
int moe_route(const void* x, const void* w_gate, int32_t dtype,
              int64_t T, int64_t H, int32_t E, int32_t k,
              const float* bias, int32_t bias_mode, int32_t renormalize,
              float* logits, int32_t* topk_idx, float* topk_w, void* stream);

/* ------------------------------------------------------------------------
 * moe_route_binarize -- a token's routing path from the predictor's output
 * (Sec. 3.2: the predictor scores every expert of every layer for each token;
 * the route r_i keeps, per layer, the experts predicted to be selected -- here
 * the k with the highest scores, the gate's own rule). Sigmoid is monotone,
 * so ranking logits ranks probabilities.
 *
 *   routes[r, j] = the expert with the j-th largest logits[r, :], descending;
 *                  equal logits go to the lower expert index; -0.0 == +0.0
 *
 * logits [rows, E] float32 DEVICE: one row per (token, layer), e.g. the
 *        [B, S, L, E] output of moe_rpp_forward viewed as [B*S*L, E]
 * routes [rows, k] uint8 DEVICE output: laid out [N, L, k] for moe_schedule
 *        when rows = N*L
 * Limits: rows >= 1, 1 <= k <= E <= 256. NaN logits: unspecified ids.
 * Errors: MOE_ERR_ARG, MOE_ERR_UNSUPPORTED, MOE_ERR_HIP.
 * ---------------------------------------------------------------------- */
int moe_route_binarize(const float* logits, int64_t rows, int32_t E, int32_t k,
                       uint8_t* routes, void* stream);

/* ------------------------------------------------------------------------
 * moe_schedule -- the Token Scheduler (Sec. 3.3): split N tokens (two adjacent
 * batches) into batches of n1 and N - n1 tokens so that few (layer, expert)
 * pairs are active per batch (Eq. 2), by the balanced two-centroid clustering
 * under routing-path similarity of Sec. 3.3.2, in exact integer form:
 *
 *   routes  [N,L,k] uint8   predicted expert ids per token and layer; the
 *                           routing path r_i has bit l*E+e set iff e appears
 *                           in routes[i,l,:]
 *   sig order   tokens ordered by their per-layer ascending expert ids, layer
 *               0 first, then by index; every tie below goes to the token
 *               earlier in this order
 *   init        m1 = least total Hamming distance to all tokens;
 *               m2 = farthest from m1
 *   assign      order tokens by d(i,m1) - d(i,m2); the first n1 are batch 1
 *   update      m_c = least summed distance to the members of batch c
 *   stop        centroids unchanged (converged) or max_iters rounds
 *   guard       keep_original_if_worse = 1: if the result activates more pairs
 *               than the input split ([0,n1), [n1,N)), return the input split
 *
 * perm    [N] int32      batch 1's token ids ascending, then batch 2's
 * demand  [2,L,E] int32  tokens of each new batch using (l, e); may be NULL
 * info    [8] int64      {iters, converged, medoid1, medoid2, obj_before,
 *                         obj_after, used_original, n1}
 * err     int32          may be NULL; set to 1 (never cleared: the caller
 *                        clears it) when the result is not to be trusted
 * Untrusted result: the rounds of larger inputs run in one launch whose
 *   blocks wait for each other at grid barriers; every wait is bounded, and a
 *   wait that gives up (after 2^20 polls, when the device kept some blocks
 *   from becoming resident that long) lets the launch finish with info[0] =
 *   -1 and *err = 1. perm, demand and the batch sizes are then unspecified.
 * Limits: N >= 1, 0 <= n1 <= N, L >= 1, 1 <= k <= E <= 256, max_iters >= 1,
 *   N < 2^26, L*E < 2^24. n1 == 0 or n1 == N returns the identity with iters = 0.
 * ---------------------------------------------------------------------- */
size_t moe_schedule_workspace(int64_t N, int32_t L, int32_t E, int32_t k);
int moe_schedule(const uint8_t* routes, int64_t N, int32_t L, int32_t E, int32_t k,
                 int64_t n1, int32_t max_iters, int32_t keep_original_if_worse,
                 int32_t* perm, int32_t* demand, int64_t* info, int32_t* err,
                 void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * moe_schedule_multi -- B-way rebatching by recursive bisection with
 * moe_schedule (an extension: Sec. 3.3.1 states the problem, Eq. 2, for two
 * batches). A node holds n tokens, in the order its parent's split left them,
 * bound for b batches; b == 1 is a batch. Otherwise moe_schedule splits the
 * node's tokens (re-indexed 0..n-1 in that order) with n1 = n*(b/2)/b
 * (integer division): its batch 1, in perm order, becomes the left child with
 * b/2 batches, its batch 2 the right child with b - b/2. The root holds all
 * N tokens in index order and B batches; the batches are the leaves, left to
 * right, so their sizes depend on N and B only.
 *
 * routes         [N,L,k] uint8   as for moe_schedule
 * perm           [N] int32       the batches' token ids, batch 0 first
 * batch_offsets  [B+1] int32     batch j is perm[batch_offsets[j] ..
 *                                batch_offsets[j+1])
 * demand         [B,L,E] int32   tokens of each batch using (l, e); may be NULL
 * info           [B-1,8] int64   moe_schedule's info of each split in
 *                                pre-order (medoids are node-local indices);
 *                                a split of an empty node records
 *                                {0, 1, -1, -1, 0, 0, 0, 0}; may be NULL
 * err            int32           as for moe_schedule: set to 1 when any split's
 *                                result is not to be trusted (its info[0] is
 *                                -1); may be NULL
 * All arrays are DEVICE memory owned by the caller; the workspace (size from
 * moe_schedule_multi_workspace, 256-byte aligned) is scratch for the call.
 * Runs B-1 two-way splits on `stream`, with no host synchronisation.
 * Limits: those of moe_schedule, and 1 <= B <= 4096 (B > N gives empty
 *   batches). Errors: MOE_ERR_ARG, MOE_ERR_UNSUPPORTED, MOE_ERR_WORKSPACE, or
 *   the first error of a split (later splits are then not launched).
 * ---------------------------------------------------------------------- */
size_t moe_schedule_multi_workspace(int64_t N, int32_t L, int32_t E, int32_t k, int32_t B);
int moe_schedule_multi(const uint8_t* routes, int64_t N, int32_t L, int32_t E, int32_t k,
                       int32_t B, int32_t max_iters, int32_t keep_original_if_worse,
                       int32_t* perm, int32_t* batch_offsets, int32_t* demand, int64_t* info,
                       int32_t* err, void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * moe_kv_gather -- KV-cache Merge and the row movement of Reindex (Sec. 3.3.3).
 * Rebatching moves tokens between batches; the KV state each token carries
 * follows it. Merge aggregates the original batches' caches in global token
 * order (source 0's tokens, then source 1's, ...); Reindex places global token
 * index[p] at new position p.
 *
 * sources[b]        DEVICE pointer: source b's cache, [L, source_tokens[b], row_bytes]
 *                   (the pointer array itself is HOST memory, n_sources <= 16)
 * index [n_out]     DEVICE int32 global token ids, or NULL for the merge itself
 *                   (then n_out must equal the total token count)
 * dst               DEVICE [L, n_out, row_bytes]: dst[l][p] = merged[l][index[p]]
 * err               DEVICE int32, set to 1 if an index is out of range (that row
 *                   is not written); the caller clears it
 * Rows move in 16-byte pieces when row_bytes and every pointer allow, else bytes.
 * Errors: MOE_ERR_ARG (missing pointer, n_sources outside 1..16, sizes < 0).
 * ---------------------------------------------------------------------- */
int moe_kv_gather(const void* const* sources, const int64_t* source_tokens, int32_t n_sources,
                  int64_t L, int64_t row_bytes, const int32_t* index, int64_t n_out, void* dst,
                  int32_t* err, void* stream);

/* ------------------------------------------------------------------------
 * moe_kv_reindex -- the index maps of Reindex (Sec. 3.3.3): new position p of
 * batch b (batch_offsets[b] <= p < batch_offsets[b+1]) holds global token
 * perm[p]; for every global token g, batch_of[g] = its new batch and pos_of[g]
 * = its position there (either output may be NULL, not both).
 * perm [N], batch_offsets [B+1] (as moe_schedule_multi writes them), batch_of
 * and pos_of [N]: DEVICE int32. err as for moe_kv_gather (a perm entry outside
 * 0..N-1). Limits: 1 <= N < 2^31, B >= 1.
 * ---------------------------------------------------------------------- */
int moe_kv_reindex(const int32_t* perm, int64_t N, const int32_t* batch_offsets, int32_t B,
                   int32_t* batch_of, int32_t* pos_of, int32_t* err, void* stream);

/* ------------------------------------------------------------------------
 * moe_stack_forward -- one batch through a stack of L MoE blocks with a
 * residual connection (Sec. 2.1's blocks, attention left out):
 *   x_l = h                                    (pre_norm = 0)
 *   x_l = h / sqrt(mean(h^2) + eps) * norm_l   (pre_norm = 1: RMS pre-norm, as
 *         in the MoE blocks of the models of Table 1; fp32, rounded once)
 *   h <- h + MoE_l(x_l),  l = 0..L-1,
 * each block moe_route -> moe_permute -> moe_expert_ffn on x_l, then
 * moe_combine with accumulate = 1 into h (h is rounded once per layer).
 *
 * h [n_tokens, H]   DEVICE, updated in place; the batch is rows token_ids[0..T)
 *                   (or rows 0..T when token_ids is NULL, then n_tokens == T)
 * w_router, w_gate, w_up, w_down   HOST arrays of L DEVICE pointers: layer l's
 *                   router [E, H] and expert slots [S, F, H], [S, F, H], [S, H, F]
 * slot_of_expert    DEVICE int32 [L, E] (-1 = not resident: those choices are
 *                   skipped) or NULL (every expert resident, S == E)
 * norm_weight       HOST array of L DEVICE pointers to [H] (dtype), or NULL
 *                   (unit weights); must be NULL when pre_norm = 0
 * h_trace           DEVICE [L, 2, T, H] or NULL: per layer the batch's state and
 *                   the block's input x_l
 * idx_trace         DEVICE int32 [L, T, k] or NULL: each layer's top-k experts
 * err               DEVICE int32, set to 1 on an out-of-range token id
 * Runs on `stream` with no host synchronisation; the workspace comes from
 * moe_stack_workspace (256-byte aligned). Limits: those of the four stages;
 * H * element size a multiple of 16 and h, h_trace 16-byte aligned.
 * Errors: MOE_ERR_ARG, MOE_ERR_UNSUPPORTED, MOE_ERR_WORKSPACE, or the first
 * error of a stage (later layers are then not launched).
 * ---------------------------------------------------------------------- */
size_t moe_stack_workspace(int64_t T, int64_t H, int64_t F, int32_t E, int32_t k, int32_t dtype);
int moe_stack_forward(void* h, int32_t dtype, int64_t n_tokens, int64_t H,
                      const int32_t* token_ids, int64_t T, int32_t L, int32_t E, int32_t k,
                      int64_t F, const void* const* w_router, const void* const* w_gate,
                      const void* const* w_up, const void* const* w_down,
                      const int32_t* slot_of_expert, int32_t S, int32_t renormalize,
                      int32_t pre_norm, const void* const* norm_weight, float eps,
                      void* h_trace, int32_t* idx_trace, int32_t* err, void* workspace,
                      size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * moe_rpp_forward -- forward pass of the routing path predictor (Sec. 3.2): a
 * T5-style encoder-decoder over B sequences of S token ids whose L heads give
 * every token logits over the E experts of each MoE layer;
 * probs = sigmoid(logits), laid out [B, S, L, E].
 *   encoder   x = emb[ids]; per layer x += Attn(rms(x)) (bidirectional, T5
 *             relative-position bias), x += W2 relu(W1 rms(x)); enc = rms(x)
 *   decoder   y = emb[ids]; per layer y += Attn(rms(y)) (causal, its own
 *             bias), y += CrossAttn(rms(y), enc), y += W2 relu(W1 rms(y));
 *             logits = rms(y) . heads^T
 *   rms(v) = v / sqrt(mean(v^2) + eps) * scale; attention without the
 *   1/sqrt(d_kv) factor; relative buckets as T5's (num_buckets, max_distance
 *   powers of two), the logarithmic ones evaluated exactly.
 * weights  DEVICE float32, moe_rpp_weights_count(dims) values in this order
 *          (linear layers [out, in]): emb [V,d]; enc_rel [nb,h]; per encoder
 *          layer ln1 [d], q, k, v, o [d,d], ln2 [d], wi [dff,d], wo [d,dff];
 *          enc_ln [d]; dec_rel [nb,h]; per decoder layer ln1 [d], q, k, v, o,
 *          ln2 [d], cq, ck, cv, co [d,d], ln3 [d], wi [dff,d], wo [d,dff];
 *          dec_ln [d]; heads [L*E, d]
 * ids      DEVICE int32 [B, S]; an id outside 0..vocab-1 sets *err (DEVICE
 *          int32, cleared by the caller) and embeds as zeros
 * probs    DEVICE float32 [B, S, L, E]; logits the same or NULL
 * Limits: d_model % n_heads == 0 with d_kv in {4, 8, 16, 32, 64};
 *   (2*S*d_kv + 2*S)*4 bytes <= 64 KiB; num_buckets even; the bucket sizes powers of two.
 * Errors: MOE_ERR_ARG, MOE_ERR_UNSUPPORTED, MOE_ERR_WORKSPACE.
 * ---------------------------------------------------------------------- */
typedef struct moe_rpp_dims {
  int32_t vocab, d_model, n_heads, d_ff, n_enc, n_dec, L, E, num_buckets, max_distance;
  float eps;
} moe_rpp_dims;
size_t moe_rpp_weights_count(const moe_rpp_dims* dims);
size_t moe_rpp_workspace(int32_t B, int32_t S, const moe_rpp_dims* dims);
int moe_rpp_forward(const int32_t* ids, int32_t B, int32_t S, const moe_rpp_dims* dims,
                    const float* weights, float* probs, float* logits, int32_t* err,
                    void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Measured ceilings (for roofline reports; not part of the method):
 * moe_probe_mfma_bf16 runs iters (a multiple of 4) rounds of 8 independent
 * 32x32x16 bf16 MFMAs per wave, 4 waves per SIMD on every compute unit, with
 * operands taken from src (DEVICE, >= 8 x 64 x 8 bf16 values, cycled so they
 * keep changing) and one float per thread written to out (DEVICE, out_len >=
 * 1024 x compute units); returns the flops launched (negative on error).
 * moe_probe_read reads `bytes` (a multiple of 16, 16-byte aligned DEVICE
 * memory) once with one 16-byte load per lane, grid-stride, and writes one
 * word per thread to out (out_len >= 2048 x compute units).
 * moe_probe_copy copies `bytes` (a multiple of 16) from src to dst (16-byte
 * aligned DEVICE buffers that do not overlap) with one 16-byte load and store
 * per lane, grid-stride.
 * ---------------------------------------------------------------------- */
int64_t moe_probe_mfma_bf16(const void* src, int64_t iters, float* out, int32_t out_len,
                            void* stream);
int moe_probe_read(const void* src, int64_t bytes, uint32_t* out, int32_t out_len,
                   void* stream);
int moe_probe_copy(const void* src, void* dst, int64_t bytes, void* stream);

/* ------------------------------------------------------------------------
 * moe_permute -- group the (token, choice) pairs of one batch by expert so
 * that every expert sees its tokens as one contiguous block of rows: the
 * batched evaluation of the selected experts E_i(x) of Sec. 2.1's MoE layer
 * (each expert applied once to all the tokens that chose it).
 *
 * Batch position i (0 <= i < T) is token t_i = token_ids[i] (or i when
 * token_ids is NULL); pair p = i*k + j is its j-th choice, on expert
 * e_p = topk_idx[t_i, j].
 *   expert_offsets[e]  = number of pairs on experts < e    ([E+1] int32 out)
 *   row_of_pair[p]     = expert_offsets[e_p] + number of pairs p' < p on e_p
 *                        (stable)                           ([T*k] int32 out)
 *   pair_of_row[r]     = the inverse map                    ([T*k] int32 out)
 *   x_perm[row(p), :]  = x[t_i, :] bit for bit              ([T*k,H] out)
 * x        [n_tokens,H] dtype; x and x_perm may both be NULL (maps only)
 * topk_idx [n_tokens,k] int32, indexed by token id
 * Limits: T >= 1, 1 <= k <= E <= 256, token ids < n_tokens, T*k < 2^31,
 *   bf16 needs H % 8 == 0, f32 needs H % 4 == 0.
 * ---------------------------------------------------------------------- */
size_t moe_permute_workspace(int64_t T, int32_t k, int32_t E);
int moe_permute(const void* x, int32_t dtype, int64_t H, int64_t n_tokens,
                const int32_t* token_ids, int64_t T,
                const int32_t* topk_idx, int32_t k, int32_t E,
                int32_t* expert_offsets, int32_t* row_of_pair, int32_t* pair_of_row,
                void* x_perm, void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * moe_permute_noalloc -- moe_permute for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation): the same computation, outputs and argument rules,
 * without a workspace argument. Its scratch is a static device array of
 * MOE_PERMUTE_NOALLOC_SCRATCH_BYTES inside the library; every device the
 * library runs on holds its own copy until the process ends. The first call
 * on a device looks up that copy's address (with the device current) and
 * keeps it; no call allocates or frees anything.
 * Every call on one device shares that device's array and leaves its contents
 * behind (nothing in it needs clearing: each call writes every word it reads):
 * calls that may overlap on one device -- on different streams, or from
 * different threads without ordering -- race and must not be issued; calls on
 * one stream are ordered and safe.
 * Limit: moe_permute_workspace(T, k, E) <= MOE_PERMUTE_NOALLOC_SCRATCH_BYTES
 *   (4 MiB: about 33.5 million tokens with E = 8, k = 2; 2.2 million with
 *   E = 60, k = 4; 262016 with E = 256, k = 8); a larger call returns
 *   MOE_ERR_WORKSPACE and enqueues nothing. MOE_ERR_HIP if the array's
 *   address cannot be looked up.
 * ---------------------------------------------------------------------- */
#define MOE_PERMUTE_NOALLOC_SCRATCH_BYTES (4 * 1024 * 1024)
int moe_permute_noalloc(const void* x, int32_t dtype, int64_t H, int64_t n_tokens,
                        const int32_t* token_ids, int64_t T,
                        const int32_t* topk_idx, int32_t k, int32_t E,
                        int32_t* expert_offsets, int32_t* row_of_pair, int32_t* pair_of_row,
                        void* x_perm, void* stream);

/* ------------------------------------------------------------------------
 * moe_expert_ffn -- the experts E_i of Sec. 2.1 in SwiGLU form, over the rows
 * each expert owns, for experts resident in the expert cache (Sec. 3.4):
 *
 *   for e with s = slot_of_expert[e] >= 0, rows r in [offsets[e], offsets[e+1]):
 *     a[r,:]      = silu(x_perm[r,:] . w_gate[s]^T) * (x_perm[r,:] . w_up[s]^T)
 *     y_perm[r,:] = a[r,:] . w_down[s]^T
 *   silu(u) = u / (1 + exp(-u)); float32 accumulation; for bf16 the
 *   activation a is rounded to bf16 before the down projection and y_perm is
 *   rounded to bf16. Rows of experts with slot < 0 (cache misses) are left
 *   untouched.
 *
 * x_perm         [max_rows,H] dtype
 * expert_offsets [E+1] int32 non-decreasing, expert_offsets[E] <= max_rows
 * slot_of_expert [E] int32, values < S (or -1); NULL means expert e uses slot
 *                e (then S >= E)
 * w_gate, w_up   [S,F,H] dtype;  w_down [S,H,F] dtype
 * y_perm         [max_rows,H] dtype output
 * Shared (always-on) experts use the same call with E = 1, offsets {0, T},
 * slot {0} and their weights concatenated along F.
 * workspace      moe_expert_ffn_workspace(max_rows, H, F, E, dtype) bytes,
 *                256-byte aligned, caller-owned: the activation a, tile
 *                counters and (bf16 with H, F multiples of 32) fp32 partial
 *                tiles of the last round of tiles, which is split along K;
 *                pieces are summed in a fixed order, so results do not depend
 *                on scheduling. Calls that share a workspace must not overlap.
 * Limits: max_rows >= 1, H >= 1, F >= 1, 1 <= E <= 256, S >= 0; bf16 needs
 *   H % 8 == 0 and F % 8 == 0.
 * ---------------------------------------------------------------------- */
size_t moe_expert_ffn_workspace(int64_t max_rows, int64_t H, int64_t F, int32_t E,
                                int32_t dtype);
int moe_expert_ffn(const void* x_perm, int32_t dtype, int64_t max_rows,
                   int64_t H, int64_t F,
                   const int32_t* expert_offsets, int32_t E,
                   const int32_t* slot_of_expert, int32_t S,
                   const void* w_gate, const void* w_up, const void* w_down,
                   void* y_perm, void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * moe_combine -- the weighted sum of Sec. 2.1, y = sum_j w_j E_{idx_j}(x),
 * over resident experts, plus always-on shared experts:
 *
 *   acc = sum_{j ascending, slot(idx[t_i,j]) >= 0} topk_w[t_i,j] * y_perm[row_of_pair[i*k+j]]
 *       + y_shared[i]                     (if y_shared != NULL)
 *       + y[t_i]                          (if accumulate)
 *   y[t_i] = acc                          (float32 accumulation, one rounding)
 *   incomplete[i] = 1 if some choice of token t_i is not resident, else 0
 *
 * y_perm [rows,H] dtype; y_shared [T,H] dtype by batch position (may be NULL)
 * topk_idx [n_tokens,k] int32, topk_w [n_tokens,k] float32, by token id
 * row_of_pair [T*k] int32 (from moe_permute); slot_of_expert [E] or NULL
 *   (all resident; E is then not needed and may be 0)
 * y [n_tokens,H] dtype: rows t_i written, other rows untouched
 * incomplete [T] int32 or NULL
 * Limits: T >= 1, k >= 1, rows >= 1, token ids < n_tokens; bf16 needs
 *   H % 8 == 0, f32 needs H % 4 == 0.
 * ---------------------------------------------------------------------- */
int moe_combine(const void* y_perm, int32_t dtype, int64_t H, int64_t rows,
                const int32_t* token_ids, int64_t T, int64_t n_tokens, int32_t k,
                const int32_t* topk_idx, const float* topk_w,
                const int32_t* row_of_pair, const int32_t* slot_of_expert, int32_t E,
                const void* y_shared, int32_t accumulate, void* y,
                int32_t* incomplete, void* stream);

/* ------------------------------------------------------------------------
 * Expert cache engine (Sec. 3.4). Host-side planning over small integer
 * tables, and the loading of whole experts into device cache slots.
 *
 * moe_plan_slots -- the resident set of one layer from predicted demand
 *   (the planning step of PLEC, Sec. 3.4.1: the cache holds the experts the
 *   prediction says the layer will use most): the S experts with the largest
 *   demand, equal demand lower expert id first, occupy slots 0..S-1 in
 *   ascending expert id; every other expert gets slot -1 (not resident).
 *   demand [E] int32 HOST; slot_of_expert [E] int32 HOST output. S larger
 *   than E is taken as E, S <= 0 leaves nothing resident. Errors: MOE_ERR_ARG
 *   on NULL or E < 1.
 *
 * moe_plec_order -- the load order of PLEC's cross-layer plan (Sec. 3.4.1):
 *   every (layer, expert) with predicted demand > 0, layers in execution
 *   order, larger demand first, equal demand lower expert id first.
 *   demand [L,E] int32 HOST array (tokens predicted to use expert e at
 *   layer l); items [L*E][2] int32 HOST output of (layer, expert) pairs;
 *   n_items: their number. Errors: MOE_ERR_ARG on NULL or L, E < 1.
 *
 * moe_plec_run -- one batch through all layers under a cache of `budget`
 *   slots shared by all layers: the cache is filled in load order before the
 *   first layer; when a layer has run its slots are refilled with the next
 *   items of later layers; an expert the batch actually uses (actual_demand
 *   > 0) is a hit if resident, else it is loaded at once (real-time
 *   correction, Sec. 3.4.2) into a free slot, else over an unused expert of
 *   the same layer, else over the later-layer item latest in load order
 *   (queued again), else it is served without caching. All arrays HOST:
 *   pred_demand, actual_demand [L,E] int32; prefetch [budget][2] int32 output
 *   (may be NULL with n_prefetch) = the items loaded before the first layer;
 *   hits, needed [L] int64 outputs; loads = every expert load of the batch.
 *
 * moe_plec_begin / moe_plec_layer / moe_plec_advance -- the same policy as
 *   moe_plec_run, step by step, with cache slots assigned, so that a run on
 *   the device can execute it: the caller copies each listed load (layer,
 *   expert, slot) into the cache and runs each layer with the slot table it
 *   gets. state: HOST memory of moe_plec_state_bytes(L, E, budget) bytes,
 *   owned by the caller, written by begin and updated by the other calls.
 *   Free slots are taken lowest index first.
 *   begin: the load order from pred_demand [L,E] (HOST int32) and the
 *     prefetch; loads [budget][3] int32 HOST output, n_loads their number.
 *   layer(l): layers in order, each once, after its actual demand [E] (HOST
 *     int32: rows routed to each expert) is known: hits and needed (HOST
 *     int64 outputs), the correction loads ([E][3], slot -1 = served without
 *     caching: no slot could be taken; never when budget >= E), and
 *     slot_of_expert [E] (HOST int32 output, may be NULL): the slot of every
 *     resident expert of layer l once the corrections are in, -1 otherwise.
 *   advance(l): layer l has run: its slots are freed and refilled with the
 *     next items of later layers; loads [budget][3] as for begin. The slots
 *     freed were read by layer l's experts: those loads must wait for them.
 *   Errors: MOE_ERR_ARG (NULL pointers, sizes, a too small state, layers out
 *   of order).
 *
 * moe_lru_run -- the baseline: a fixed cache of `capacity` experts per layer
 *   with least-recently-used replacement, kept across B batches; a layer's
 *   used experts are looked up in ascending id. actual_demand [B,L,E] int32
 *   HOST; hits, needed: totals (HOST int64 outputs).
 *
 * moe_load_experts -- copies whole experts into cache slots: for i < n,
 *   expert expert_ids[i] of the store (w_gate_src, w_up_src [E_store,F,H],
 *   w_down_src [E_store,H,F], dtype) into slot slot_ids[i] of the cache
 *   (w_gate, w_up [S,F,H], w_down [S,H,F] DEVICE arrays), as asynchronous
 *   copies on `stream`. expert_ids, slot_ids: HOST int32 [n]. The store is
 *   normally pinned host memory (copies from pageable memory are staged and
 *   do not overlap); any address HIP can copy from is accepted. The caller
 *   must not let kernels that read a destination slot run concurrently.
 *   Errors: MOE_ERR_ARG on NULL pointers, ids out of range or a destination
 *   slot named twice (nothing is enqueued); MOE_ERR_HIP if a copy cannot be
 *   enqueued.
 * ---------------------------------------------------------------------- */
int moe_plan_slots(const int32_t* demand, int32_t E, int32_t S, int32_t* slot_of_expert);
int moe_plec_order(const int32_t* demand, int32_t L, int32_t E, int32_t* items,
                   int32_t* n_items);
int moe_plec_run(const int32_t* pred_demand, const int32_t* actual_demand, int32_t L,
                 int32_t E, int32_t budget, int32_t* prefetch, int32_t* n_prefetch,
                 int64_t* hits, int64_t* needed, int64_t* loads);
size_t moe_plec_state_bytes(int32_t L, int32_t E, int32_t budget);
int moe_plec_begin(const int32_t* pred_demand, int32_t L, int32_t E, int32_t budget,
                   void* state, size_t state_bytes, int32_t* loads, int32_t* n_loads);
int moe_plec_layer(void* state, int32_t l, const int32_t* actual_demand,
                   int32_t* slot_of_expert, int32_t* loads, int32_t* n_loads, int64_t* hits,
                   int64_t* needed);
int moe_plec_advance(void* state, int32_t l, int32_t* loads, int32_t* n_loads);
int moe_lru_run(const int32_t* actual_demand, int32_t B, int32_t L, int32_t E,
                int32_t capacity, int64_t* hits, int64_t* needed);
int moe_load_experts(const void* w_gate_src, const void* w_up_src, const void* w_down_src,
                     int32_t E_store, void* w_gate, void* w_up, void* w_down, int32_t S,
                     int64_t H, int64_t F, int32_t dtype, const int32_t* expert_ids,
                     const int32_t* slot_ids, int32_t n, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MOEFLOW_H */
