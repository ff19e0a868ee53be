"""Thin Python binding of libmoeflow.so (include/moeflow.h).

Every function here only marshals arguments: it checks tensor placement,
dtype and shape, allocates outputs and workspaces with torch (device memory),
and passes raw pointers and the current HIP stream to the C entry point of the
same name. All arithmetic of the hot path runs in the library's HIP kernels;
there is no fallback. If the library has not been built, the first call raises.
"""
import ctypes
import os

import numpy as np

from . import build as _build

MOE_OK, MOE_ERR_ARG, MOE_ERR_UNSUPPORTED, MOE_ERR_WORKSPACE, MOE_ERR_HIP = range(5)
MOE_F32, MOE_BF16 = 0, 1

_LIB = None


class MoeError(RuntimeError):
    def __init__(self, fn, status, msg):
        super().__init__(f"{fn} failed with status {status}: {msg}")
        self.status = status


def _c_i64():
    return ctypes.c_int64


def load_library(path=None):
    """Load libmoeflow.so (once). Raises if it does not exist."""
    global _LIB
    if _LIB is not None:
        return _LIB
    path = path or _build.library_path()
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build the HIP library first "
            "(python -c 'import __graft_entry__ as g; g.build()')")
    # torch's HIP runtime first: the library's libamdhip64.so.7 then resolves
    # to it, whereas loaded the other way round torch (which names the
    # runtime without its version) brings a second runtime into the process
    # and kernel launches from one fail on the other's device state
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    sig = {
        "moe_abi_version": (I32, []),
        "moe_status_str": (ctypes.c_char_p, [ctypes.c_int]),
        "moe_route": (I32, [P, P, I32, I64, I64, I32, I32, P, I32, I32, P, P, P, P]),
        "moe_route_binarize": (I32, [P, I64, I32, I32, P, P]),
        "moe_schedule_workspace": (SZ, [I64, I32, I32, I32]),
        "moe_schedule": (I32, [P, I64, I32, I32, I32, I64, I32, I32, P, P, P, P, P, SZ, P]),
        "moe_kv_gather": (I32, [P, P, I32, I64, I64, P, I64, P, P, P]),
        "moe_kv_reindex": (I32, [P, I64, P, I32, P, P, P, P]),
        "moe_stack_workspace": (SZ, [I64, I64, I64, I32, I32, I32]),
        "moe_stack_forward": (I32, [P, I32, I64, I64, P, I64, I32, I32, I32, I64, P, P, P, P, P,
                                    I32, I32, I32, P, ctypes.c_float, P, P, P, P, SZ, P]),
        "moe_probe_mfma_bf16": (I64, [P, I64, P, I32, P]),
        "moe_probe_read": (I32, [P, I64, P, I32, P]),
        "moe_probe_copy": (I32, [P, P, I64, P]),
        "moe_rpp_weights_count": (SZ, [P]),
        "moe_rpp_workspace": (SZ, [I32, I32, P]),
        "moe_rpp_forward": (I32, [P, I32, I32, P, P, P, P, P, P, SZ, P]),
        "moe_schedule_multi_workspace": (SZ, [I64, I32, I32, I32, I32]),
        "moe_schedule_multi": (I32, [P, I64, I32, I32, I32, I32, I32, I32, P, P, P, P, P, P,
                                     SZ, P]),
        "moe_permute_workspace": (SZ, [I64, I32, I32]),
        "moe_permute": (I32, [P, I32, I64, I64, P, I64, P, I32, I32, P, P, P, P, P, SZ, P]),
        "moe_permute_noalloc": (I32, [P, I32, I64, I64, P, I64, P, I32, I32, P, P, P, P, P]),
        "moe_expert_ffn_workspace": (SZ, [I64, I64, I64, I32, I32]),
        "moe_expert_ffn": (I32, [P, I32, I64, I64, I64, P, I32, P, I32, P, P, P, P, P, SZ, P]),
        "moe_combine": (I32, [P, I32, I64, I64, P, I64, I64, I32, P, P, P, P, I32, P, I32, P,
                              P, P]),
        "moe_plan_slots": (I32, [P, I32, I32, P]),
        "moe_plec_order": (I32, [P, I32, I32, P, P]),
        "moe_plec_run": (I32, [P, P, I32, I32, I32, P, P, P, P, P]),
        "moe_lru_run": (I32, [P, I32, I32, I32, I32, P, P]),
        "moe_plec_state_bytes": (SZ, [I32, I32, I32]),
        "moe_plec_begin": (I32, [P, I32, I32, I32, P, SZ, P, P]),
        "moe_plec_layer": (I32, [P, I32, P, P, P, P, P, P]),
        "moe_plec_advance": (I32, [P, I32, P, P]),
        "moe_load_experts": (I32, [P, P, P, I32, P, P, P, I32, I64, I64, I32, P, P, I32, P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _LIB = lib
    return lib


def exported_symbols():
    return ["moe_abi_version", "moe_status_str", "moe_route", "moe_route_binarize",
            "moe_schedule_workspace",
            "moe_schedule", "moe_schedule_multi_workspace", "moe_schedule_multi",
            "moe_permute_workspace", "moe_permute", "moe_permute_noalloc",
            "moe_expert_ffn_workspace", "moe_expert_ffn", "moe_combine", "moe_kv_gather",
            "moe_kv_reindex", "moe_stack_workspace", "moe_stack_forward",
            "moe_rpp_weights_count", "moe_rpp_workspace", "moe_rpp_forward",
            "moe_probe_mfma_bf16", "moe_probe_read", "moe_probe_copy", "moe_plan_slots", "moe_plec_order",
            "moe_plec_run", "moe_lru_run", "moe_load_experts", "moe_plec_state_bytes",
            "moe_plec_begin", "moe_plec_layer", "moe_plec_advance"]


def _check(name, status):
    if status != MOE_OK:
        msg = load_library().moe_status_str(status).decode()
        raise MoeError(name, status, msg)


def _torch():
    import torch
    return torch


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return MOE_BF16
    if t.dtype == torch.float32:
        return MOE_F32
    raise TypeError(f"unsupported dtype {t.dtype}: bfloat16 or float32 expected")


def _dev(*ts):
    for t in ts:
        if t is not None:
            if not t.is_cuda:
                raise ValueError("every tensor must be on the GPU")
            if not t.is_contiguous():
                raise ValueError("every tensor must be contiguous")


def _workspace(nbytes, device, workspace):
    torch = _torch()
    if nbytes == 0:
        return None, 0
    if workspace is not None:
        if workspace.numel() * workspace.element_size() < nbytes:
            raise ValueError(f"workspace too small: {nbytes} bytes needed")
        return workspace, workspace.numel() * workspace.element_size()
    ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    ws = ws[off:off + nbytes]
    return ws, nbytes


def workspace_tensor(nbytes, device):
    """A 256-byte aligned uint8 device buffer of at least nbytes."""
    return _workspace(nbytes, device, None)[0]


# ----------------------------------------------------------------------- route
def route(x=None, w_gate=None, k=1, bias=None, renormalize=True, logits=None,
          want_logits=False, topk_idx=None, topk_w=None, stream=None):
    """moe_route. x-mode: route(x, w_gate, k, ...). logits-in mode:
    route(k=k, logits=z). Returns (topk_idx int32 [T,k], topk_w f32 [T,k],
    logits or None)."""
    torch = _torch()
    lib = load_library()
    if x is None and w_gate is None:
        if logits is None:
            raise ValueError("logits-in mode needs logits")
        _dev(logits)
        T, E = logits.shape
        dt, H, bias_mode = MOE_F32, 0, 0
        dev = logits.device
    else:
        _dev(x, w_gate, bias)
        T, H = x.shape
        E = w_gate.shape[0]
        if w_gate.shape[1] != H or w_gate.dtype != x.dtype:
            raise ValueError("w_gate must be [E, H] with the dtype of x")
        dt = _dtype_code(x)
        dev = x.device
        bias_mode = 0
        if bias is not None:
            if bias.dtype != torch.float32:
                raise TypeError("bias must be float32")
            bias_mode = 1 if bias.dim() == 1 else 2
        if logits is None and want_logits:
            logits = torch.empty((T, E), dtype=torch.float32, device=dev)
    if topk_idx is None:
        topk_idx = torch.empty((T, k), dtype=torch.int32, device=dev)
    if topk_w is None:
        topk_w = torch.empty((T, k), dtype=torch.float32, device=dev)
    st = lib.moe_route(_ptr(x), _ptr(w_gate), dt, T, H, E, k, _ptr(bias), bias_mode,
                       1 if renormalize else 0, _ptr(logits), _ptr(topk_idx), _ptr(topk_w),
                       _stream(stream))
    _check("moe_route", st)
    return topk_idx, topk_w, logits


# -------------------------------------------------------------------- schedule
def route_binarize(logits, k, routes=None, stream=None):
    """moe_route_binarize over logits float32 [..., E] (rows = the leading
    dimensions). Returns uint8 routes [..., k]."""
    torch = _torch()
    lib = load_library()
    _dev(logits, routes)
    if logits.dtype != torch.float32 or logits.dim() < 2:
        raise TypeError("logits must be float32 [..., E]")
    E = logits.shape[-1]
    rows = logits.numel() // E
    shape = tuple(logits.shape[:-1]) + (k,)
    if routes is None:
        routes = torch.empty(shape, dtype=torch.uint8, device=logits.device)
    elif routes.dtype != torch.uint8 or tuple(routes.shape) != shape:
        raise ValueError("routes must be uint8 of shape logits.shape[:-1] + (k,)")
    _check("moe_route_binarize", lib.moe_route_binarize(_ptr(logits), rows, E, k, _ptr(routes),
                                                        _stream(stream)))
    return routes


def schedule_workspace(N, L, E, k):
    return load_library().moe_schedule_workspace(N, L, E, k)


def schedule(routes, E, n1=None, max_iters=10, keep_original_if_worse=True,
             perm=None, demand=None, info=None, workspace=None, want_demand=True,
             err=None, stream=None):
    """moe_schedule over routes uint8 [N, L, k]. Returns (perm int32 [N],
    demand int32 [2, L, E] or None, info int64 [8]). err: optional device
    int32 [1] that the call sets to 1 when its result is not to be trusted."""
    torch = _torch()
    lib = load_library()
    _dev(routes)
    if routes.dtype != torch.uint8 or routes.dim() != 3:
        raise TypeError("routes must be uint8 [N, L, k]")
    N, L, k = routes.shape
    n1 = N // 2 if n1 is None else int(n1)
    dev = routes.device
    if perm is None:
        perm = torch.empty(N, dtype=torch.int32, device=dev)
    if demand is None and want_demand:
        demand = torch.empty((2, L, E), dtype=torch.int32, device=dev)
    if info is None:
        info = torch.empty(8, dtype=torch.int64, device=dev)
    ws, nbytes = _workspace(lib.moe_schedule_workspace(N, L, E, k), dev, workspace)
    _dev(err)
    st = lib.moe_schedule(_ptr(routes), N, L, E, k, n1, max_iters,
                          1 if keep_original_if_worse else 0, _ptr(perm), _ptr(demand),
                          _ptr(info), _ptr(err), _ptr(ws), nbytes, _stream(stream))
    _check("moe_schedule", st)
    return perm, demand, info


def schedule_multi_workspace(N, L, E, k, B):
    return load_library().moe_schedule_multi_workspace(N, L, E, k, B)


def schedule_multi(routes, E, B, max_iters=10, keep_original_if_worse=True, perm=None,
                   batch_offsets=None, demand=None, info=None, workspace=None,
                   want_demand=True, want_info=True, err=None, stream=None):
    """moe_schedule_multi over routes uint8 [N, L, k] into B batches. Returns
    (perm int32 [N], batch_offsets int32 [B+1], demand int32 [B, L, E] or None,
    info int64 [B-1, 8] or None). err: as for schedule."""
    torch = _torch()
    lib = load_library()
    _dev(routes)
    if routes.dtype != torch.uint8 or routes.dim() != 3:
        raise TypeError("routes must be uint8 [N, L, k]")
    N, L, k = routes.shape
    dev = routes.device
    if perm is None:
        perm = torch.empty(N, dtype=torch.int32, device=dev)
    if batch_offsets is None:
        batch_offsets = torch.empty(B + 1, dtype=torch.int32, device=dev)
    if demand is None and want_demand:
        demand = torch.empty((B, L, E), dtype=torch.int32, device=dev)
    if info is None and want_info and B > 1:
        info = torch.empty((B - 1, 8), dtype=torch.int64, device=dev)
    ws, nbytes = _workspace(lib.moe_schedule_multi_workspace(N, L, E, k, B), dev, workspace)
    _dev(err)
    st = lib.moe_schedule_multi(_ptr(routes), N, L, E, k, B, max_iters,
                                1 if keep_original_if_worse else 0, _ptr(perm),
                                _ptr(batch_offsets), _ptr(demand), _ptr(info), _ptr(err),
                                _ptr(ws), nbytes, _stream(stream))
    _check("moe_schedule_multi", st)
    return perm, batch_offsets, demand, info


# ------------------------------------------------------------------- KV cache
def kv_gather(sources, index=None, out=None, err=None, stream=None):
    """moe_kv_gather. sources: list of device tensors [L, T_b, ...] (one per
    original batch, same dtype and trailing shape); index int32 [n_out] or
    None (the merge). Returns (out [L, n_out, ...], err int32 [1])."""
    torch = _torch()
    lib = load_library()
    if not sources or len(sources) > 16:
        raise ValueError("1 to 16 sources")
    _dev(*sources, index)
    L = sources[0].shape[0]
    tail = tuple(sources[0].shape[2:])
    for s_ in sources:
        if s_.shape[0] != L or tuple(s_.shape[2:]) != tail or s_.dtype != sources[0].dtype:
            raise ValueError("sources must share L, dtype and the trailing shape")
        if not s_.is_contiguous():
            raise ValueError("sources must be contiguous")
    row_bytes = sources[0].element_size()
    for d in tail:
        row_bytes *= d
    total = sum(s_.shape[1] for s_ in sources)
    n_out = total if index is None else index.shape[0]
    dev = sources[0].device
    if out is None:
        out = torch.empty((L, n_out) + tail, dtype=sources[0].dtype, device=dev)
    if err is None:
        err = torch.zeros(1, dtype=torch.int32, device=dev)
    ptrs = (ctypes.c_void_p * len(sources))(*[s_.data_ptr() for s_ in sources])
    rows = (ctypes.c_int64 * len(sources))(*[s_.shape[1] for s_ in sources])
    st = lib.moe_kv_gather(ptrs, rows, len(sources), L, row_bytes, _ptr(index), n_out,
                           _ptr(out), _ptr(err), _stream(stream))
    _check("moe_kv_gather", st)
    return out, err


def kv_reindex(perm, batch_offsets, batch_of=None, pos_of=None, err=None, stream=None):
    """moe_kv_reindex. Returns (batch_of int32 [N], pos_of int32 [N], err)."""
    torch = _torch()
    lib = load_library()
    _dev(perm, batch_offsets)
    N = perm.shape[0]
    B = batch_offsets.shape[0] - 1
    dev = perm.device
    if batch_of is None:
        batch_of = torch.empty(N, dtype=torch.int32, device=dev)
    if pos_of is None:
        pos_of = torch.empty(N, dtype=torch.int32, device=dev)
    if err is None:
        err = torch.zeros(1, dtype=torch.int32, device=dev)
    st = lib.moe_kv_reindex(_ptr(perm), N, _ptr(batch_offsets), B, _ptr(batch_of), _ptr(pos_of),
                            _ptr(err), _stream(stream))
    _check("moe_kv_reindex", st)
    return batch_of, pos_of, err


# ------------------------------------------------------------------------- RPP
class RppDims(ctypes.Structure):
    """moe_rpp_dims."""
    _fields_ = [(n, ctypes.c_int32) for n in ("vocab", "d_model", "n_heads", "d_ff", "n_enc",
                                               "n_dec", "L", "E", "num_buckets",
                                               "max_distance")] + [("eps", ctypes.c_float)]


def rpp_dims(dims):
    return RppDims(**{k: dims[k] for k in (n for n, _ in RppDims._fields_)})


def rpp_weights_count(dims):
    return load_library().moe_rpp_weights_count(ctypes.byref(rpp_dims(dims)))


def rpp_forward(ids, weights, dims, probs=None, logits=None, err=None, workspace=None,
                want_logits=False, stream=None):
    """moe_rpp_forward. ids int32 [B, S]; weights float32 [n] (packed); dims a
    dict of moe_rpp_dims fields. Returns (probs [B, S, L, E], logits or None, err)."""
    torch = _torch()
    lib = load_library()
    _dev(ids, weights)
    if ids.dtype != torch.int32 or ids.dim() != 2 or weights.dtype != torch.float32:
        raise TypeError("ids int32 [B, S] and float32 weights")
    B, S = ids.shape
    g = rpp_dims(dims)
    if weights.numel() != lib.moe_rpp_weights_count(ctypes.byref(g)):
        raise ValueError("weights do not match the dimensions")
    dev = ids.device
    shape = (B, S, dims["L"], dims["E"])
    if probs is None:
        probs = torch.empty(shape, dtype=torch.float32, device=dev)
    if logits is None and want_logits:
        logits = torch.empty(shape, dtype=torch.float32, device=dev)
    if err is None:
        err = torch.zeros(1, dtype=torch.int32, device=dev)
    ws, nbytes = _workspace(lib.moe_rpp_workspace(B, S, ctypes.byref(g)), dev, workspace)
    st = lib.moe_rpp_forward(_ptr(ids), B, S, ctypes.byref(g), _ptr(weights), _ptr(probs),
                             _ptr(logits), _ptr(err), _ptr(ws), nbytes, _stream(stream))
    _check("moe_rpp_forward", st)
    return probs, logits, err


# ----------------------------------------------------------------------- stack
def stack_workspace(T, H, F, E, k, dtype_code=MOE_BF16):
    return load_library().moe_stack_workspace(T, H, F, E, k, dtype_code)


def stack_forward(h, layers, k, token_ids=None, slot_of_expert=None, S=None, renormalize=True,
                  pre_norm=False, norm_weights=None, eps=1e-5, h_trace=None, idx_trace=None,
                  err=None, workspace=None, stream=None):
    """moe_stack_forward: the batch (rows token_ids of h, or all rows) through
    the layers, h updated in place. layers: list of (w_router [E,H], w_gate
    [S,F,H], w_up [S,F,H], w_down [S,H,F]) device tensors; norm_weights: list
    of [H] tensors or None (unit weights, with pre_norm). Returns (h, err)."""
    torch = _torch()
    lib = load_library()
    _dev(h, token_ids, slot_of_expert, h_trace, idx_trace)
    n_tokens, H = h.shape
    T = token_ids.shape[0] if token_ids is not None else n_tokens
    L = len(layers)
    E = layers[0][0].shape[0]
    Sw, F, _ = layers[0][1].shape
    S = Sw if S is None else S
    dt = _dtype_code(h)
    for lay in layers:
        _dev(*lay)
        if (tuple(lay[0].shape) != (E, H) or tuple(lay[1].shape) != (Sw, F, H)
                or tuple(lay[2].shape) != (Sw, F, H) or tuple(lay[3].shape) != (Sw, H, F)):
            raise ValueError("every layer must be router [E,H], w_gate/w_up [S,F,H], w_down [S,H,F]")
        if any(t.dtype != h.dtype or not t.is_contiguous() for t in lay):
            raise ValueError("layer weights must be contiguous with the dtype of h")
    if err is None:
        err = torch.zeros(1, dtype=torch.int32, device=h.device)
    arr = lambda j: (ctypes.c_void_p * L)(*[lay[j].data_ptr() for lay in layers])
    nw = None
    if norm_weights is not None:
        if not pre_norm or len(norm_weights) != L:
            raise ValueError("norm_weights needs pre_norm and one [H] tensor per layer")
        _dev(*norm_weights)
        if any(tuple(w_.shape) != (H,) or w_.dtype != h.dtype for w_ in norm_weights):
            raise ValueError("norm weights must be [H] with the dtype of h")
        nw = (ctypes.c_void_p * L)(*[w_.data_ptr() for w_ in norm_weights])
    ws, nbytes = _workspace(lib.moe_stack_workspace(T, H, F, E, k, dt), h.device, workspace)
    st = lib.moe_stack_forward(_ptr(h), dt, n_tokens, H, _ptr(token_ids), T, L, E, k, F, arr(0),
                               arr(1), arr(2), arr(3), _ptr(slot_of_expert), S,
                               1 if renormalize else 0, 1 if pre_norm else 0, nw, float(eps),
                               _ptr(h_trace), _ptr(idx_trace), _ptr(err), _ptr(ws), nbytes,
                               _stream(stream))
    _check("moe_stack_forward", st)
    return h, err


# --------------------------------------------------------------------- permute
def permute_workspace(T, k, E):
    return load_library().moe_permute_workspace(T, k, E)


def permute(x, topk_idx, E, token_ids=None, T=None, expert_offsets=None, row_of_pair=None,
            pair_of_row=None, x_perm=None, workspace=None, stream=None):
    """moe_permute. x [n_tokens, H] (or None for maps only), topk_idx
    [n_tokens, k]; the batch is token_ids (or every row). Returns
    (expert_offsets [E+1], row_of_pair [T*k], pair_of_row [T*k], x_perm)."""
    torch = _torch()
    lib = load_library()
    _dev(x, topk_idx, token_ids)
    n_tokens, k = topk_idx.shape
    if T is None:
        T = token_ids.shape[0] if token_ids is not None else n_tokens
    dev = topk_idx.device
    P = T * k
    if expert_offsets is None:
        expert_offsets = torch.empty(E + 1, dtype=torch.int32, device=dev)
    if row_of_pair is None:
        row_of_pair = torch.empty(P, dtype=torch.int32, device=dev)
    if pair_of_row is None:
        pair_of_row = torch.empty(P, dtype=torch.int32, device=dev)
    dt, H = MOE_F32, 0
    if x is not None:
        dt, H = _dtype_code(x), x.shape[1]
        if x_perm is None:
            x_perm = torch.empty((P, H), dtype=x.dtype, device=dev)
    ws, nbytes = _workspace(lib.moe_permute_workspace(T, k, E), dev, workspace)
    st = lib.moe_permute(_ptr(x), dt, H, x.shape[0] if x is not None else n_tokens,
                         _ptr(token_ids), T, _ptr(topk_idx), k, E, _ptr(expert_offsets),
                         _ptr(row_of_pair), _ptr(pair_of_row), _ptr(x_perm), _ptr(ws), nbytes,
                         _stream(stream))
    _check("moe_permute", st)
    return expert_offsets, row_of_pair, pair_of_row, x_perm


def permute_noalloc(x, topk_idx, E, expert_offsets, row_of_pair, pair_of_row, x_perm=None,
                    token_ids=None, T=None, stream=None):
    """moe_permute_noalloc: moe_permute into outputs the caller allocated
    beforehand, with the library's static scratch instead of a workspace
    (nothing is allocated). Calls that may overlap on one device race."""
    lib = load_library()
    _dev(x, topk_idx, token_ids, expert_offsets, row_of_pair, pair_of_row, x_perm)
    n_tokens, k = topk_idx.shape
    if T is None:
        T = token_ids.shape[0] if token_ids is not None else n_tokens
    if (x is None) != (x_perm is None):
        raise ValueError("x and x_perm go together")
    if (expert_offsets.numel() < E + 1 or row_of_pair.numel() < T * k
            or pair_of_row.numel() < T * k):
        raise ValueError("output maps too small")
    dt, H = MOE_F32, 0
    if x is not None:
        dt, H = _dtype_code(x), x.shape[1]
        if x_perm.dtype != x.dtype or x_perm.shape[1] != H or x_perm.shape[0] < T * k:
            raise ValueError("x_perm must be [T*k, H] of x's dtype")
    st = lib.moe_permute_noalloc(_ptr(x), dt, H, x.shape[0] if x is not None else n_tokens,
                                 _ptr(token_ids), T, _ptr(topk_idx), k, E,
                                 _ptr(expert_offsets), _ptr(row_of_pair), _ptr(pair_of_row),
                                 _ptr(x_perm), _stream(stream))
    _check("moe_permute_noalloc", st)
    return expert_offsets, row_of_pair, pair_of_row, x_perm


# ------------------------------------------------------------------ expert ffn
def expert_ffn_workspace(max_rows, H, F, E, dtype_code=MOE_BF16):
    return load_library().moe_expert_ffn_workspace(max_rows, H, F, E, dtype_code)


def expert_ffn(x_perm, expert_offsets, w_gate, w_up, w_down, slot_of_expert=None,
               y_perm=None, workspace=None, stream=None):
    """moe_expert_ffn. x_perm [max_rows, H]; w_gate/w_up [S, F, H]; w_down
    [S, H, F]; expert_offsets [E+1]. Rows of non-resident experts of y_perm are
    left as they were. Returns y_perm."""
    torch = _torch()
    lib = load_library()
    _dev(x_perm, expert_offsets, w_gate, w_up, w_down, slot_of_expert)
    max_rows, H = x_perm.shape
    S, F, H2 = w_gate.shape
    if H2 != H or tuple(w_up.shape) != (S, F, H) or tuple(w_down.shape) != (S, H, F):
        raise ValueError("weights must be w_gate/w_up [S,F,H] and w_down [S,H,F]")
    if not (w_gate.dtype == w_up.dtype == w_down.dtype == x_perm.dtype):
        raise TypeError("weights and activations must share one dtype")
    E = expert_offsets.shape[0] - 1
    dt = _dtype_code(x_perm)
    if y_perm is None:
        y_perm = torch.empty_like(x_perm)
    ws, nbytes = _workspace(lib.moe_expert_ffn_workspace(max_rows, H, F, E, dt),
                            x_perm.device, workspace)
    st = lib.moe_expert_ffn(_ptr(x_perm), dt, max_rows, H, F, _ptr(expert_offsets), E,
                            _ptr(slot_of_expert), S, _ptr(w_gate), _ptr(w_up), _ptr(w_down),
                            _ptr(y_perm), _ptr(ws), nbytes, _stream(stream))
    _check("moe_expert_ffn", st)
    return y_perm


# --------------------------------------------------------------------- combine
def combine(y_perm, topk_idx, topk_w, row_of_pair, token_ids=None, slot_of_expert=None,
            y_shared=None, y=None, accumulate=False, want_incomplete=True, incomplete=None,
            stream=None):
    """moe_combine. Returns (y [n_tokens, H], incomplete int32 [T] or None)."""
    torch = _torch()
    lib = load_library()
    _dev(y_perm, topk_idx, topk_w, row_of_pair, token_ids, slot_of_expert, y_shared, y)
    rows, H = y_perm.shape
    n_tokens, k = topk_idx.shape
    T = token_ids.shape[0] if token_ids is not None else n_tokens
    E = slot_of_expert.shape[0] if slot_of_expert is not None else 0
    dev = y_perm.device
    if y is None:
        if accumulate:
            raise ValueError("accumulate needs an existing y")
        y = torch.zeros((n_tokens, H), dtype=y_perm.dtype, device=dev)
    if incomplete is None and want_incomplete:
        incomplete = torch.empty(T, dtype=torch.int32, device=dev)
    st = lib.moe_combine(_ptr(y_perm), _dtype_code(y_perm), H, rows, _ptr(token_ids), T,
                         y.shape[0], k, _ptr(topk_idx), _ptr(topk_w), _ptr(row_of_pair),
                         _ptr(slot_of_expert), E, _ptr(y_shared), 1 if accumulate else 0,
                         _ptr(y), _ptr(incomplete), _stream(stream))
    _check("moe_combine", st)
    return y, incomplete


# ------------------------------------------------------------------ slot table
def plan_slots(demand, S):
    """moe_plan_slots: the resident set of one layer from predicted demand
    int [E] (host). Returns slot_of_expert int32 [E] (-1 = not resident)."""
    lib = load_library()
    d = np.ascontiguousarray(np.asarray(demand), dtype=np.int32)
    if d.ndim != 1:
        raise ValueError("demand must be [E]")
    slot = np.empty(d.shape[0], dtype=np.int32)
    _check("moe_plan_slots", lib.moe_plan_slots(d.ctypes.data_as(ctypes.c_void_p), d.shape[0],
                                                int(S), slot.ctypes.data_as(ctypes.c_void_p)))
    return slot


# ------------------------------------------------------------- expert cache
def _host_i32(a):
    a = np.ascontiguousarray(a, dtype=np.int32)
    return a, a.ctypes.data_as(ctypes.c_void_p)


def plec_order(demand):
    """moe_plec_order over demand int [L, E] (host). Returns int32 [n, 2]
    (layer, expert) in load order."""
    lib = load_library()
    d, dp = _host_i32(demand)
    L, E = d.shape
    items = np.empty((L * E, 2), dtype=np.int32)
    n = ctypes.c_int32(0)
    _check("moe_plec_order", lib.moe_plec_order(dp, L, E, items.ctypes.data_as(ctypes.c_void_p),
                                                ctypes.byref(n)))
    return items[:n.value]


def plec_run(pred_demand, actual_demand, budget):
    """moe_plec_run: one batch under a shared cache of `budget` slots. Returns
    dict(prefetch int32 [n, 2], hits int64 [L], needed int64 [L], loads)."""
    lib = load_library()
    p, pp = _host_i32(pred_demand)
    a, ap = _host_i32(actual_demand)
    if p.shape != a.shape:
        raise ValueError("pred_demand and actual_demand must both be [L, E]")
    L, E = p.shape
    pre = np.empty((max(int(budget), 1), 2), dtype=np.int32)
    npre = ctypes.c_int32(0)
    hits = np.empty(L, dtype=np.int64)
    needed = np.empty(L, dtype=np.int64)
    loads = ctypes.c_int64(0)
    st = lib.moe_plec_run(pp, ap, L, E, int(budget), pre.ctypes.data_as(ctypes.c_void_p),
                          ctypes.byref(npre), hits.ctypes.data_as(ctypes.c_void_p),
                          needed.ctypes.data_as(ctypes.c_void_p), ctypes.byref(loads))
    _check("moe_plec_run", st)
    return {"prefetch": pre[:npre.value], "hits": hits, "needed": needed, "loads": loads.value}


class PlecPlanner:
    """moe_plec_begin / moe_plec_layer / moe_plec_advance over host state:
    the PLEC policy step by step with cache slots assigned. Loads come back as
    int32 [n, 3] rows (layer, expert, slot)."""

    def __init__(self, pred_demand, budget):
        self.lib = load_library()
        d, dp = _host_i32(pred_demand)
        self.L, self.E = d.shape
        self.budget = int(budget)
        n = self.lib.moe_plec_state_bytes(self.L, self.E, self.budget)
        self.state = ctypes.create_string_buffer(n)
        self._buf = np.empty((max(self.budget, self.E, 1), 3), dtype=np.int32)
        cnt = ctypes.c_int32(0)
        _check("moe_plec_begin", self.lib.moe_plec_begin(
            dp, self.L, self.E, self.budget, self.state, n,
            self._buf.ctypes.data_as(ctypes.c_void_p), ctypes.byref(cnt)))
        self.prefetch = self._buf[:cnt.value].copy()

    def layer(self, l, actual_demand):
        """Returns (slot_of_expert int32 [E], correction loads [n, 3], hits,
        needed)."""
        a, ap = _host_i32(actual_demand)
        slot = np.empty(self.E, dtype=np.int32)
        cnt = ctypes.c_int32(0)
        hits, needed = ctypes.c_int64(0), ctypes.c_int64(0)
        _check("moe_plec_layer", self.lib.moe_plec_layer(
            self.state, int(l), ap, slot.ctypes.data_as(ctypes.c_void_p),
            self._buf.ctypes.data_as(ctypes.c_void_p), ctypes.byref(cnt), ctypes.byref(hits),
            ctypes.byref(needed)))
        return slot, self._buf[:cnt.value].copy(), hits.value, needed.value

    def advance(self, l):
        """Layer l has run: returns the refill loads [n, 3]."""
        cnt = ctypes.c_int32(0)
        _check("moe_plec_advance", self.lib.moe_plec_advance(
            self.state, int(l), self._buf.ctypes.data_as(ctypes.c_void_p), ctypes.byref(cnt)))
        return self._buf[:cnt.value].copy()


def lru_run(actual_demands, capacity):
    """moe_lru_run over actual_demands int [B, L, E]: returns (hits, needed)."""
    lib = load_library()
    a, ap = _host_i32(actual_demands)
    B, L, E = a.shape
    hits, needed = ctypes.c_int64(0), ctypes.c_int64(0)
    _check("moe_lru_run", lib.moe_lru_run(ap, B, L, E, int(capacity), ctypes.byref(hits),
                                          ctypes.byref(needed)))
    return hits.value, needed.value


def load_experts(store, cache, expert_ids, slot_ids, stream=None):
    """moe_load_experts: store = (w_gate, w_up, w_down) tensors [E_store, ...]
    (normally pinned host memory), cache = the same three on the device
    [S, ...]; copies expert expert_ids[i] into slot slot_ids[i] on `stream`."""
    lib = load_library()
    sg, su, sd = store
    cg, cu, cd = cache
    E_store, F, H = sg.shape
    S = cg.shape[0]
    if sd.shape != (E_store, H, F) or cd.shape != (S, H, F) or cg.shape != (S, F, H):
        raise ValueError("store [E,F,H],[E,F,H],[E,H,F] and cache [S,F,H],[S,F,H],[S,H,F]")
    _dev(cg, cu, cd)
    for t in (sg, su, sd):
        if not t.is_contiguous() or t.dtype != cg.dtype:
            raise ValueError("store tensors must be contiguous and of the cache's dtype")
    e, ep = _host_i32(expert_ids)
    s, sp = _host_i32(slot_ids)
    if e.shape != s.shape:
        raise ValueError("expert_ids and slot_ids must have the same length")
    st = lib.moe_load_experts(_ptr(sg), _ptr(su), _ptr(sd), E_store, _ptr(cg), _ptr(cu),
                              _ptr(cd), S, H, F, _dtype_code(cg), ep, sp, int(e.shape[0]),
                              _stream(stream))
    _check("moe_load_experts", st)
