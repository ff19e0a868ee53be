"""Token Scheduler (TS) of Sec. 3.3, written out in integers.

Routing path (Sec. 3.2 and Sec. 3.3.1): token i's route is a binary matrix
r_i in {0,1}^{L x E}, r_i[l, e] = 1 iff expert e is among the k experts the
token uses at layer l.

Objective (Sec. 3.3.1, Eq. 2): split the N = 2T tokens into two batches and
minimise sum_{l,e} (R_1[l,e] + R_2[l,e]) where R_c is the element-wise OR of the
routes in batch c, i.e. the number of (layer, expert) pairs each batch activates.

Approximation (Sec. 3.3.2): a K-means-style clustering into two equal-size
groups under the similarity S_ij = 1 - d_ij / (L E), d_ij the Hamming distance
of the two routes; each token goes to the closest cluster, and each centroid
becomes the member token with the highest mean similarity to its own cluster;
this repeats until it settles or an iteration limit is reached.

Because S_ij is a decreasing affine function of d_ij, "most similar" is
"smallest Hamming distance" and the whole procedure stays in integers. The
points the paper leaves open are fixed as follows (every one is a reading):

  1. Batch sizes: batch 1 gets n1 tokens (default N // 2), batch 2 the rest.
  2. Signature order: key_i is the concatenation over layers l = 0..L-1 of the
     ascending expert ids token i uses at layer l; tokens are ordered by key,
     lexicographically (layer 0 most significant), equal keys by token index.
     sig_rank_i is the position in that order. Every later tie is broken by the
     lower sig_rank, which keeps tokens with identical routes adjacent.
  3. Initial centroids: m1 = the token with the least total distance to all
     tokens; m2 = the token farthest from m1 (i != m1).
  4. Assignment under the equal-size constraint: delta_i = d(i,m1) - d(i,m2);
     tokens ordered by (delta_i, sig_rank_i); the first n1 form batch 1.
     For two fixed centres and fixed batch sizes this ordering minimises the
     summed distance of tokens to their own centre.
  5. Centroid update: m_c = argmin over i in batch c of sum_{j in batch c} d_ij
     (j = i included), i.e. the member with the highest mean similarity.
  6. Stop when (m1, m2) does not change (converged) or after max_iters
     assignment/update rounds; the split returned is the last assignment.
  7. Guard (not in the paper; keep_original_if_worse): if the result activates
     more (layer, expert) pairs than the original split ([0,n1), [n1,N)), the
     original split is returned.
  8. Output: perm lists batch 1's tokens in ascending index, then batch 2's.
     demand[c, l, e] counts the tokens of batch c whose route uses (l, e).
     info = [iters, converged, medoid1, medoid2, obj_before, obj_after,
             used_original, n1].

The distance sums use the expansion of the Hamming distance of 0/1 vectors,
d(a, b) = |a| + |b| - 2 <a, b>, summed over a cluster; tests pin it against
pairwise XOR counts. Pinned in tests/test_oracle_schedule.py (worked example of
Sec. 3.3, brute-force optimum, planted clusters, fixed point, identities).
"""
import numpy as np


def route_bits(routes, E):
    """routes: int [N, L, k] expert ids -> int64 0/1 array [N, L, E]."""
    routes = np.asarray(routes, dtype=np.int64)
    N, L, k = routes.shape
    r = np.zeros((N, L, E), dtype=np.int64)
    for j in range(k):
        np.put_along_axis(r, routes[:, :, j:j + 1], 1, axis=2)
    return r


def eq2_objective(bits, in_batch1):
    """Eq. 2: number of active (layer, expert) pairs of batch 1 plus batch 2.

    bits: [N, L*E] (or [N, L, E]) 0/1; in_batch1: bool [N]."""
    b = np.asarray(bits, dtype=np.int64).reshape(len(in_batch1), -1)
    m = np.asarray(in_batch1, dtype=bool)
    r1 = b[m].any(axis=0) if m.any() else np.zeros(b.shape[1], bool)
    r2 = b[~m].any(axis=0) if (~m).any() else np.zeros(b.shape[1], bool)
    return int(r1.sum()) + int(r2.sum())


def signature_rank(routes):
    """sig_rank[i] = position of token i when tokens are ordered by their
    layer-by-layer sorted expert ids (layer 0 most significant), ties by index."""
    routes = np.asarray(routes, dtype=np.int64)
    N = routes.shape[0]
    keys = np.sort(routes, axis=2).reshape(N, -1)
    # np.lexsort sorts by the LAST key first and is stable, so passing the
    # columns in reverse makes column 0 the most significant; stability leaves
    # equal keys in index order.
    order = np.lexsort(tuple(keys[:, c] for c in range(keys.shape[1] - 1, -1, -1)))
    rank = np.empty(N, dtype=np.int64)
    rank[order] = np.arange(N, dtype=np.int64)
    return rank


def hamming_to(bits, m):
    """d(i, m) for every token i. bits: [N, LE] 0/1."""
    b = np.asarray(bits, dtype=np.int64)
    return (b != b[m][None, :]).sum(axis=1).astype(np.int64)


def cluster_distance_sums(bits, members):
    """For each i in members: sum_{j in members} d_ij, in members' order."""
    b = np.asarray(bits, dtype=np.int64)[np.asarray(members, dtype=np.int64)]
    size = b.shape[0]
    ones = b.sum(axis=1)            # |r_i|
    col = b.sum(axis=0)             # c_b = sum_j r_jb
    return size * ones + ones.sum() - 2 * (b @ col)


def _argmin_by(values, sig, cand):
    """The candidate with the smallest value, ties to the lower sig_rank."""
    cand = np.asarray(cand, dtype=np.int64)
    o = np.lexsort((sig[cand], values))
    return int(cand[o[0]])


def schedule(routes, E, n1=None, max_iters=10, keep_original_if_worse=True):
    """Returns (perm int64 [N], demand int64 [2, L, E], info int64 [8])."""
    routes = np.asarray(routes, dtype=np.int64)
    N, L, k = routes.shape
    if n1 is None:
        n1 = N // 2
    r3 = route_bits(routes, E)
    bits = r3.reshape(N, L * E)
    sig = signature_rank(routes)
    original = np.arange(N) < n1
    obj_before = eq2_objective(bits, original)

    iters, converged, used_original = 0, 1, 0
    med = (-1, -1)
    in1 = original.copy()
    if 0 < n1 < N:
        everyone = np.arange(N)
        m1 = _argmin_by(cluster_distance_sums(bits, everyone), sig, everyone)
        d1 = hamming_to(bits, m1)
        others = everyone[everyone != m1]
        m2 = _argmin_by(-d1[others], sig, others)
        converged = 0
        for it in range(1, max_iters + 1):
            iters = it
            delta = hamming_to(bits, m1) - hamming_to(bits, m2)
            order = np.lexsort((sig, delta))
            in1 = np.zeros(N, dtype=bool)
            in1[order[:n1]] = True
            med = (m1, m2)
            c1 = np.nonzero(in1)[0]
            c2 = np.nonzero(~in1)[0]
            m1_new = _argmin_by(cluster_distance_sums(bits, c1), sig, c1)
            m2_new = _argmin_by(cluster_distance_sums(bits, c2), sig, c2)
            if (m1_new, m2_new) == (m1, m2):
                converged = 1
                break
            m1, m2 = m1_new, m2_new
    obj_after = eq2_objective(bits, in1)
    if keep_original_if_worse and obj_after > obj_before:
        in1 = original
        obj_after = obj_before
        used_original = 1
    perm = np.concatenate([np.nonzero(in1)[0], np.nonzero(~in1)[0]]).astype(np.int64)
    demand = np.stack([r3[in1].sum(axis=0), r3[~in1].sum(axis=0)]).astype(np.int64)
    info = np.array([iters, converged, med[0], med[1], obj_before, obj_after,
                     used_original, n1], dtype=np.int64)
    return perm, demand, info


def multi_batch_offsets(N, B):
    """Batch boundaries of the B-way split of N tokens by recursive bisection:
    a set of n tokens bound for b batches puts n * (b // 2) // b of them
    (floor) into the first b // 2 batches and the rest into the other
    b - b // 2. Returns int64 [B + 1]."""
    sizes = []

    def rec(n, b):
        if b == 1:
            sizes.append(n)
            return
        bl = b // 2
        n1 = n * bl // b
        rec(n1, bl)
        rec(n - n1, b - bl)

    rec(int(N), int(B))
    return np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)


def schedule_multi(routes, E, B, max_iters=10, keep_original_if_worse=True):
    """B-way rebatching by recursive bisection with the two-way scheduler
    above (an extension: Sec. 3.3.1 states the problem for two batches).

    A node holds n tokens (in the order its parent's split left them) and the
    number b of batches they form. b == 1 is a batch. Otherwise the two-way
    scheduler runs on the node's tokens, re-indexed 0..n-1 in that order, with
    n1 = n * (b // 2) // b; its batch 1 (in its perm order) becomes the left
    child with b // 2 batches, its batch 2 the right child with the rest. The
    batches are the leaves from left to right.

    Returns (perm int64 [N]: the leaves' tokens concatenated,
             offsets int64 [B + 1],
             demand int64 [B, L, E]: tokens of each batch using (l, e),
             info int64 [B - 1, 8]: the two-way info of each split in
                 pre-order (medoids are node-local indices); a split of an
                 empty node records [0, 1, -1, -1, 0, 0, 0, 0]).
    """
    routes = np.asarray(routes, dtype=np.int64)
    N, L, k = routes.shape
    infos = []

    def rec(ids, b):
        if b == 1:
            return [ids]
        bl = b // 2
        n = len(ids)
        n1 = n * bl // b
        if n == 0:
            infos.append(np.array([0, 1, -1, -1, 0, 0, 0, 0], dtype=np.int64))
            return rec(ids, bl) + rec(ids, b - bl)
        p, _, info = schedule(routes[ids], E, n1, max_iters, keep_original_if_worse)
        infos.append(info)
        ids = ids[p]
        return rec(ids[:n1], bl) + rec(ids[n1:], b - bl)

    leaves = rec(np.arange(N, dtype=np.int64), int(B))
    perm = np.concatenate(leaves).astype(np.int64)
    offsets = np.concatenate([[0], np.cumsum([len(x) for x in leaves])]).astype(np.int64)
    r3 = route_bits(routes, E)
    demand = np.stack([r3[x].sum(axis=0) for x in leaves]).astype(np.int64)
    info = np.stack(infos) if infos else np.zeros((0, 8), dtype=np.int64)
    return perm, offsets, demand, info


def batch_accuracy(true_bits, pred_bits):
    """Batch-level accuracy of Sec. 4.3.3: the per-layer share of the experts a
    batch really activates that the prediction also activates, averaged over
    layers. Inputs are token routes [n, L, E] (0/1); both are OR-ed over the
    batch first. Layers the batch does not activate at all are skipped."""
    R = np.asarray(true_bits).astype(bool).any(axis=0)
    Rh = np.asarray(pred_bits).astype(bool).any(axis=0)
    den = R.sum(axis=1)
    num = (R & Rh).sum(axis=1)
    ok = den > 0
    return float(np.mean(num[ok] / den[ok]))
