"""Softmax top-k gating (Sec. 2.1 of the paper: the gate scores are the softmax
of the router projection x.W_g, the k experts with the highest scores are
selected, and the layer output weights each selected expert by its score).

Readings taken where the paper is silent:
  * W_g is stored as [E, H] (one row per expert), so x.W_g of the paper is
    x @ W_g.T here. An optional bias is added to the logits: none, one value per
    expert ([E]) or one per token and expert ([T, E]).
  * Selection order: descending logit; equal logits go to the lower expert
    index. -0.0 and +0.0 compare equal. NaN logits are outside the contract.
  * renormalize=1 divides the selected scores by their sum (the gates then sum
    to one); renormalize=0 keeps the raw softmax scores G_i(x), as written in
    Sec. 2.1.
Pinned in tests/test_oracle_gating.py by brute-force ranking, the closed form
of the renormalised gates, and the E=1 / k=E special cases.
"""
import numpy as np


def router_logits(x, w_gate, bias=None):
    """z[t, e] = sum_h x[t, h] * W_g[e, h] (+ bias), in float64.

    x: [T, H]; w_gate: [E, H]; bias: None, [E] or [T, E].
    """
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w_gate, dtype=np.float64)
    z = x @ w.T
    if bias is not None:
        b = np.asarray(bias, dtype=np.float64)
        z = z + (b[None, :] if b.ndim == 1 else b)
    return z


def topk_select(z, k):
    """Indices of the k largest logits of each row, in descending logit order,
    equal logits ordered by ascending expert index. Returns int64 [T, k]."""
    z = np.asarray(z, dtype=np.float64)
    # A stable sort of the negated logits keeps equal values in index order.
    order = np.argsort(-z, axis=1, kind="stable")
    return order[:, :k].astype(np.int64)


def softmax(z):
    """Row-wise softmax over all E experts (the gate G(x) of Sec. 2.1)."""
    z = np.asarray(z, dtype=np.float64)
    m = z.max(axis=1, keepdims=True)
    e = np.exp(z - m)
    return e / e.sum(axis=1, keepdims=True)


def gate_weights(z, idx, renormalize=True):
    """Scores of the selected experts: G_{idx}(x), optionally divided by their
    sum. z: [T, E]; idx: [T, k]. Returns float64 [T, k]."""
    p = softmax(z)
    w = np.take_along_axis(p, np.asarray(idx, dtype=np.int64), axis=1)
    if renormalize:
        w = w / w.sum(axis=1, keepdims=True)
    return w


def route(x, w_gate, k, bias=None, renormalize=True):
    """Full gating step: (logits [T,E], idx [T,k] int64, weights [T,k] f64)."""
    z = router_logits(x, w_gate, bias)
    idx = topk_select(z, k)
    return z, idx, gate_weights(z, idx, renormalize)
