"""KV-cache Merge and Reindex of Sec. 3.3.3 (adaptive KV-cache management),
written out as array indexing. Test infrastructure: only tests, the smoke check
and the benchmark's CPU baseline use it.

Rebatching moves tokens between the two batches of a scheduling unit, so the
KV state each token carries must follow it:

  Merge    the per-batch caches of the original batches are aggregated into
           one cache in global token order: the original batches' tokens one
           after another (batch 0 first), each batch in its own order;
  Reindex  every token gets its place in the new layout: new position p
           (batch b covers positions offsets[b] .. offsets[b+1]-1) holds global
           token perm[p], and each global token g knows its new batch and its
           position inside it.

A cache is an array [L, T, C]: L layers, T tokens, C values per token and
layer (keys and values of every head over the token's context, flattened; the
layout inside C is opaque here).
"""
import numpy as np


def kv_merge(sources):
    """sources: list of [L, T_b, C] arrays of the original batches. Returns
    [L, sum T_b, C] in global token order."""
    return np.concatenate([np.asarray(s) for s in sources], axis=1)


def kv_gather(merged, index):
    """Reindexed cache: out[l, p] = merged[l, index[p]]."""
    return np.asarray(merged)[:, np.asarray(index, dtype=np.int64), :]


def kv_reindex(perm, offsets):
    """perm [N]: new position -> global token; offsets [B+1]: batch bounds.
    Returns (batch_of [N], pos_of [N]) indexed by global token id."""
    perm = np.asarray(perm, dtype=np.int64)
    offsets = np.asarray(offsets, dtype=np.int64)
    N = perm.shape[0]
    batch_of = np.empty(N, dtype=np.int64)
    pos_of = np.empty(N, dtype=np.int64)
    for b in range(len(offsets) - 1):
        span = perm[offsets[b]:offsets[b + 1]]
        batch_of[span] = b
        pos_of[span] = np.arange(len(span))
    return batch_of, pos_of
