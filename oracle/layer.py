"""The composed MoE layer of Sec. 2.1 (gate, expert evaluation, weighted sum),
over one batch and one resident set, plus the dense FFN that a one-expert
top-1 layer must reduce to (the pin of the whole composition), and a stack of
such layers with a residual connection between them."""
import numpy as np

from .gating import route
from .permute import permute
from .ffn import expert_ffn, swiglu
from .combine import combine


def dense_ffn(x, w_gate, w_up, w_down):
    return swiglu(x, w_gate, w_up, w_down)


def moe_layer(x, w_router, k, w_gate, w_up, w_down, bias=None, renormalize=True,
              slot_of_expert=None, token_ids=None, shared=None):
    """x: [n, H]; experts stored per slot: w_gate/w_up [S, F, H], w_down
    [S, H, F]. shared = (wg, wu, wd) of the always-on shared experts
    concatenated along F, or None. Returns a dict of every intermediate."""
    x = np.asarray(x, dtype=np.float64)
    E = np.asarray(w_router).shape[0]
    if slot_of_expert is None:
        slot_of_expert = np.arange(E)
    z, idx, w = route(x, w_router, k, bias, renormalize)
    offsets, rop, por, xp = permute(x, idx, E, token_ids)
    yp, computed = expert_ffn(xp, offsets, slot_of_expert, w_gate, w_up, w_down)
    tok = np.arange(x.shape[0]) if token_ids is None else np.asarray(token_ids)
    ys = None if shared is None else swiglu(x[tok], *shared)
    y, inc = combine(np.nan_to_num(yp), idx, w, rop, token_ids, slot_of_expert,
                     ys, n_out=x.shape[0])
    return dict(logits=z, idx=idx, w=w, offsets=offsets, row_of_pair=rop,
                pair_of_row=por, x_perm=xp, y_perm=yp, computed=computed,
                y_shared=ys, y=y, incomplete=inc)


def round_bf16(a):
    """Round float64 values to the nearest bfloat16 value (8 significant bits,
    ties to even), returned as float64. Normal range only (|a| >= 2^-126)."""
    u = np.ascontiguousarray(a, dtype=np.float64).view(np.uint64)
    drop = np.uint64(45)                         # 52 - 7 fraction bits dropped
    lsb = (u >> drop) & np.uint64(1)
    r = (u + (np.uint64(1) << np.uint64(44)) - np.uint64(1) + lsb) >> drop << drop
    return r.view(np.float64)


def rms_norm(h, weight=None, eps=1e-5):
    """Root-mean-square normalisation of each row (the pre-norm of the MoE
    blocks of Table 1's models): h / sqrt(mean(h^2) + eps) * weight."""
    h = np.asarray(h, dtype=np.float64)
    r = h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps)
    return r if weight is None else r * np.asarray(weight, dtype=np.float64)


def moe_stack(h, layers, k, renormalize=True, pre_norm=False, eps=1e-5):
    """A stack of MoE blocks with a residual connection (the transformer blocks
    of Sec. 2.1 with the attention half left out): x_l = h_l, or with pre_norm
    x_l = bf16(rms_norm(h_l, norm_l)); h_{l+1} = h_l + y_l, y_l the MoE layer's
    output on x_l. The state between layers is stored in bfloat16 (h_{l+1}
    rounded once), as the HIP path stores it.

    layers: list of dicts with w_router [E, H], w_gate/w_up [S, F, H], w_down
    [S, H, F], optionally slot_of_expert [E] and norm [H]. Returns (h_L,
    states [L, n, H], inputs [L, n, H], idx [L, n, k])."""
    h = np.asarray(h, dtype=np.float64)
    states, ins, idxs = [], [], []
    for lay in layers:
        states.append(h)
        x = round_bf16(rms_norm(h, lay.get("norm"), eps)) if pre_norm else h
        ins.append(x)
        out = moe_layer(x, lay["w_router"], k, lay["w_gate"], lay["w_up"], lay["w_down"],
                        renormalize=renormalize, slot_of_expert=lay.get("slot_of_expert"))
        idxs.append(out["idx"])
        h = round_bf16(h + out["y"])
    return h, np.stack(states), np.stack(ins), np.stack(idxs)
