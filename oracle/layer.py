"""The composed MoE layer of Sec. 2.1 (gate, expert evaluation, weighted sum),
over one batch and one resident set, plus the dense FFN that a one-expert
top-1 layer must reduce to (the pin of the whole composition)."""
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
