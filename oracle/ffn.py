"""The expert E_i(x) of Sec. 2.1, in the gated-SiLU (SwiGLU) form used by the
Mixtral-, Qwen-MoE- and DeepSeek-shaped models of Table 1:

    E(x) = W_down . ( silu(W_gate . x) * (W_up . x) ),   silu(u) = u / (1 + e^-u)

with W_gate, W_up: [F, H] and W_down: [H, F]. Everything is float64 with no
intermediate rounding. Experts that the slot table marks as not resident
(slot < 0) are not evaluated: their rows are cache misses (Sec. 3.4).

Pinned in tests/test_oracle_ffn.py against a pure-Python loop version and by
the dense-FFN identity of a one-expert top-1 layer.
"""
import math

import numpy as np


def silu(u):
    u = np.asarray(u, dtype=np.float64)
    return u / (1.0 + np.exp(-u))


def swiglu(x, w_gate, w_up, w_down):
    """x: [M, H] -> [M, H] through one SwiGLU expert (matrix form)."""
    x = np.asarray(x, dtype=np.float64)
    h1 = x @ np.asarray(w_gate, dtype=np.float64).T
    h3 = x @ np.asarray(w_up, dtype=np.float64).T
    return (silu(h1) * h3) @ np.asarray(w_down, dtype=np.float64).T


def swiglu_loops(x, w_gate, w_up, w_down):
    """The same expert written as explicit scalar loops (used to pin swiglu)."""
    M, H = len(x), len(x[0])
    F = len(w_gate)
    out = [[0.0] * H for _ in range(M)]
    for m in range(M):
        a = []
        for f in range(F):
            g = 0.0
            u = 0.0
            for h in range(H):
                g += float(w_gate[f][h]) * float(x[m][h])
                u += float(w_up[f][h]) * float(x[m][h])
            a.append(g / (1.0 + math.exp(-g)) * u)
        for h in range(H):
            s = 0.0
            for f in range(F):
                s += float(w_down[h][f]) * a[f]
            out[m][h] = s
    return np.array(out, dtype=np.float64)


def expert_ffn(x_perm, offsets, slot_of_expert, w_gate, w_up, w_down):
    """Apply expert e (weights in slot slot_of_expert[e]) to rows
    [offsets[e], offsets[e+1]) of x_perm.

    Returns (y_perm float64 [R, H], computed bool [R]); rows of non-resident
    experts are left as NaN and flagged False.
    """
    x_perm = np.asarray(x_perm, dtype=np.float64)
    offsets = np.asarray(offsets, dtype=np.int64)
    E = len(offsets) - 1
    R, H = x_perm.shape[0], x_perm.shape[1]
    y = np.full((R, H), np.nan, dtype=np.float64)
    computed = np.zeros(R, dtype=bool)
    for e in range(E):
        s = int(slot_of_expert[e])
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if s < 0 or hi == lo:
            continue
        y[lo:hi] = swiglu(x_perm[lo:hi], w_gate[s], w_up[s], w_down[s])
        computed[lo:hi] = True
    return y, computed
