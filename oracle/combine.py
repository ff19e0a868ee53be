"""Weighted combine of Sec. 2.1, y = sum over selected experts of G_i(x) E_i(x),
restricted to the experts that are resident in the expert cache; a token with a
selected expert that is not resident is flagged incomplete (the misprediction
case that real-time correction handles, Sec. 3.4). Always-on shared experts,
when present, are added with weight one.

Pinned in tests/test_oracle_layer.py (k=E soft-MoE identity, shared-expert
concatenation, resident + missed parts summing to the full output).
"""
import numpy as np


def combine(y_perm, idx, w, row_of_pair, token_ids=None, slot_of_expert=None,
            y_shared=None, n_out=None, y_init=None):
    """Returns (y float64 [n_out, H], incomplete int64 [T]).

    Token t_i (= token_ids[i] or i) receives
        y[t_i] = (y_init[t_i] if given) + sum_{j resident} w[t_i, j] * y_perm[row(i*k+j)]
                 + (y_shared[i] if given)
    Rows of y not named by token_ids are zero (or y_init).
    """
    idx = np.asarray(idx, dtype=np.int64)
    w = np.asarray(w, dtype=np.float64)
    y_perm = np.asarray(y_perm, dtype=np.float64)
    k = idx.shape[1]
    tok = (np.arange(idx.shape[0]) if token_ids is None
           else np.asarray(token_ids, dtype=np.int64))
    T = tok.shape[0]
    H = y_perm.shape[1]
    if n_out is None:
        n_out = idx.shape[0]
    y = (np.zeros((n_out, H)) if y_init is None
         else np.array(y_init, dtype=np.float64, copy=True))
    incomplete = np.zeros(T, dtype=np.int64)
    for i in range(T):
        t = tok[i]
        acc = np.zeros(H)
        for j in range(k):
            e = idx[t, j]
            if slot_of_expert is not None and slot_of_expert[e] < 0:
                incomplete[i] = 1
                continue
            acc += w[t, j] * y_perm[row_of_pair[i * k + j]]
        if y_shared is not None:
            acc += np.asarray(y_shared[i], dtype=np.float64)
        y[t] = y[t] + acc
    return y, incomplete
