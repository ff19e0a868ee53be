"""Expert-major grouping of (token, choice) pairs.

Sec. 2.1 evaluates each selected expert E_i on the tokens routed to it; running
an expert once over all of its tokens needs those tokens gathered into one
contiguous block per expert. This module states that grouping directly:

  * a batch position i (0 <= i < T) holds token t_i = token_ids[i] (or i);
  * pair p = i*k + j is the j-th choice of that token, on expert e_p = idx[t_i, j];
  * counts[e] = number of pairs on expert e; offsets = exclusive prefix sum;
  * row(p) = offsets[e_p] + number of earlier pairs p' < p on the same expert
    (a stable grouping: rows of one expert keep the pair order);
  * pair_of_row is the inverse map, and x_perm[row(p)] = x[t_i].

Pinned in tests/test_oracle_permute.py (bijection, count sum T*k, stability,
row contents, equality with a library stable sort).
"""
import numpy as np


def permute(x, idx, E, token_ids=None):
    """Returns (offsets [E+1], row_of_pair [T*k], pair_of_row [T*k], x_perm).

    x: [n_tokens, H] (any dtype; rows copied exactly); idx: [n_tokens, k];
    token_ids: None or [T] rows of x / idx forming the batch.
    """
    idx = np.asarray(idx, dtype=np.int64)
    k = idx.shape[1]
    if token_ids is None:
        tok = np.arange(idx.shape[0], dtype=np.int64)
    else:
        tok = np.asarray(token_ids, dtype=np.int64)
    T = tok.shape[0]
    P = T * k
    expert_of_pair = np.empty(P, dtype=np.int64)
    for i in range(T):
        for j in range(k):
            expert_of_pair[i * k + j] = idx[tok[i], j]
    counts = np.zeros(E, dtype=np.int64)
    for p in range(P):
        counts[expert_of_pair[p]] += 1
    offsets = np.zeros(E + 1, dtype=np.int64)
    for e in range(E):
        offsets[e + 1] = offsets[e] + counts[e]
    seen = np.zeros(E, dtype=np.int64)
    row_of_pair = np.empty(P, dtype=np.int64)
    for p in range(P):
        e = expert_of_pair[p]
        row_of_pair[p] = offsets[e] + seen[e]
        seen[e] += 1
    pair_of_row = np.empty(P, dtype=np.int64)
    pair_of_row[row_of_pair] = np.arange(P, dtype=np.int64)
    x = np.asarray(x)
    x_perm = np.empty((P,) + x.shape[1:], dtype=x.dtype)
    for p in range(P):
        x_perm[row_of_pair[p]] = x[tok[p // k]]
    return offsets, row_of_pair, pair_of_row, x_perm
