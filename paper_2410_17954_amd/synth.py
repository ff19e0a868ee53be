"""Seeded synthetic inputs for the MoE-layer hot path.

This module only draws inputs; it contains none of the method's arithmetic
(no gating, grouping, expert evaluation or scheduling). Both the GPU path and
the CPU checker consume exactly the arrays it returns.

Recipe (every stream is a numpy PCG64 generator spawned from
SeedSequence(seed), one child per named tensor, so each tensor is independent
of the sizes of the others):
  * hidden states x ~ N(0, 1); router and expert weights ~ N(0, 0.02);
    drawn in float32, then rounded to bfloat16 (round to nearest even) for the
    bf16 workloads. bf16 tensors are returned as uint16 bit patterns. Large
    tensors are drawn in blocks along their first axis (1024 rows of x, one
    expert of a weight stack), block b from the stream (seed, tensor, b).
  * Zipf-skewed router bias (Qwen- and DeepSeek-shaped layers): expert e gets
    b_e = ln(rho_e^-s / sum_e' rho_e'^-s), rho = 1 + a seeded permutation of
    0..E-1, so the softmax odds of expert e are scaled by its Zipf mass.
  * predicted routes over L layers (route-grouped workloads): layer 0 draws k
    distinct experts by Zipf(s) over a seeded per-layer popularity order;
    at layer l > 0 choice j keeps the expert of layer l-1 with probability
    `keep` when that id is still free, and otherwise draws Zipf(s) over the
    experts not yet chosen at layer l.
  * optional coupling of the real router to the prediction: a per-token bias
    of `boost` on the experts predicted for the layer being run.
These stand in for the paper's models (Table 1) and datasets, which are not
available; the shapes follow Table 1's Mixtral, Qwen1.5-MoE and DeepSeek rows.
"""
import concurrent.futures
import os

import numpy as np

# Workload shapes, by name. T = tokens in one layer call, H hidden, E routed
# experts, F expert FFN width, k experts per token, S resident slots, n_shared
# always-on shared experts (each of width F), L layers in the predicted route;
# seed is the seed its inputs are drawn with.
WORKLOADS = {
    "tiny_fp32": dict(seed=1, dtype="f32", T=64, H=128, E=8, F=256, k=2, S=8,
            n_shared=0, L=4, keep=0.7, zipf=1.1, zipf_bias=None, boost=0.0),
    "mixtral8x7b_layer": dict(seed=2, dtype="bf16", T=4096, H=4096, E=8, F=14336,
            k=2, S=8, n_shared=0, L=32, keep=0.7, zipf=1.1, zipf_bias=None,
            boost=0.0),
    "mixtral8x7b_route_grouped": dict(seed=3, dtype="bf16", T=8192, H=4096, E=8,
            F=14336, k=2, S=4, n_shared=0, L=32, keep=0.7, zipf=1.1,
            zipf_bias=None, boost=3.0),
    "qwen15_moe_layer": dict(seed=4, dtype="bf16", T=8192, H=2048, E=60, F=1408,
            k=4, S=32, n_shared=4, L=24, keep=0.7, zipf=1.2, zipf_bias=1.2,
            boost=0.0),
    "deepseek_v2_lite_layer": dict(seed=5, dtype="bf16", T=32768, H=2048, E=64,
            F=1408, k=6, S=48, n_shared=2, L=26, keep=0.7, zipf=1.0,
            zipf_bias=1.0, boost=3.0),
}

# Child-stream index of every named tensor (fixed forever: changing it
# changes every seeded input).
_STREAM = {"x": 0, "router": 1, "w_gate": 2, "w_up": 3, "w_down": 4,
           "shared_gate": 5, "shared_up": 6, "shared_down": 7,
           "bias_rank": 8, "routes": 9, "logits": 10, "idx": 11, "misc": 12}


def workload(name):
    return dict(WORKLOADS[name], name=name)


def rng_for(seed, name, block=None):
    """Generator of the named tensor (and of one block of it along axis 0)."""
    key = [int(seed), _STREAM[name]] + ([] if block is None else [int(block)])
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(key)))


def bf16_bits(a):
    """float32 array -> uint16 bfloat16 bit patterns, round to nearest even
    (finite inputs)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    out = np.empty(a.shape, dtype=np.uint16)
    flat_in = a.reshape(-1).view(np.uint32)
    flat_out = out.reshape(-1)
    step = 1 << 22
    for lo in range(0, flat_in.size, step):
        u = flat_in[lo:lo + step]
        r = (u >> 16) & 1
        r += 0x7FFF
        r += u
        r >>= 16
        flat_out[lo:lo + step] = r
    return out


def bf16_to_f32(bits):
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def values(arr):
    """Exact float64 values of a stored tensor (uint16 = bf16 bit patterns)."""
    if arr.dtype == np.uint16:
        return bf16_to_f32(arr).astype(np.float64)
    return np.asarray(arr, dtype=np.float64)


_POOL_THREADS = min(16, os.cpu_count() or 1)


def _normal(seed, name, shape, std, dtype, rows_per_block=1):
    """N(0, std^2) draws of `shape`, in blocks of `rows_per_block` along axis 0,
    block b drawn from its own stream (seed, name, b); threads only change
    the speed, never the values."""
    n0 = shape[0]
    inner = shape[1:]
    out = np.empty(shape, dtype=np.uint16 if dtype == "bf16" else np.float32)
    blocks = list(range(0, n0, rows_per_block))

    def fill(lo):
        g = rng_for(seed, name, lo // rows_per_block)
        hi = min(n0, lo + rows_per_block)
        a = g.standard_normal(size=(hi - lo,) + tuple(inner), dtype=np.float32)
        if std != 1.0:
            a *= np.float32(std)
        out[lo:hi] = bf16_bits(a) if dtype == "bf16" else a

    if len(blocks) == 1:
        fill(0)
    else:
        with concurrent.futures.ThreadPoolExecutor(_POOL_THREADS) as ex:
            list(ex.map(fill, blocks))
    return out


def layer_inputs(cfg, seed, T=None, parts=("x", "router", "experts", "shared", "bias")):
    """Draw the tensors of one MoE layer. Returns a dict of numpy arrays:
    x [T,H], w_router [E,H], w_gate/w_up [E,F,H], w_down [E,H,F],
    shared_gate/shared_up [n_s*F,H], shared_down [H,n_s*F], bias [E] (f32)."""
    T = cfg["T"] if T is None else T
    H, E, F, dt = cfg["H"], cfg["E"], cfg["F"], cfg["dtype"]
    out = {}
    if "x" in parts:
        out["x"] = _normal(seed, "x", (T, H), 1.0, dt, rows_per_block=1024)
    if "router" in parts:
        out["w_router"] = _normal(seed, "router", (E, H), 0.02, dt, rows_per_block=E)
    if "experts" in parts:
        out["w_gate"] = _normal(seed, "w_gate", (E, F, H), 0.02, dt)
        out["w_up"] = _normal(seed, "w_up", (E, F, H), 0.02, dt)
        out["w_down"] = _normal(seed, "w_down", (E, H, F), 0.02, dt)
    if "shared" in parts and cfg.get("n_shared", 0) > 0:
        Fs = cfg["n_shared"] * F
        out["shared_gate"] = _normal(seed, "shared_gate", (Fs, H), 0.02, dt, rows_per_block=F)
        out["shared_up"] = _normal(seed, "shared_up", (Fs, H), 0.02, dt, rows_per_block=F)
        out["shared_down"] = _normal(seed, "shared_down", (H, Fs), 0.02, dt, rows_per_block=H)
    if "bias" in parts and cfg.get("zipf_bias") is not None:
        out["bias"] = zipf_bias(E, cfg["zipf_bias"], popularity_order(seed, E, 1)[0])
    return out


def popularity_order(seed, E, L):
    """Per-layer popularity: order[l, r] = expert id of rank r at layer l."""
    g = rng_for(seed, "bias_rank")
    return np.stack([g.permutation(E) for _ in range(L)]).astype(np.int64)


def zipf_bias(E, s, order):
    """b[order[r]] = ln((r+1)^-s / sum_r' (r'+1)^-s) as float32 [E]."""
    mass = np.arange(1, E + 1, dtype=np.float64) ** (-float(s))
    mass /= mass.sum()
    b = np.empty(E, dtype=np.float64)
    b[np.asarray(order)] = np.log(mass)
    return b.astype(np.float32)


def predicted_routes(N, L, E, k, keep, s, seed):
    """Markov-chain predicted routes, uint8 [N, L, k] (k distinct ids per layer)."""
    if E > 256:
        raise ValueError("routes are stored as uint8: E must be <= 256")
    g = rng_for(seed, "routes")
    order = popularity_order(seed, E, L)
    mass = np.arange(1, E + 1, dtype=np.float64) ** (-float(s))
    routes = np.zeros((N, L, k), dtype=np.int64)
    rows = np.arange(N)
    for l in range(L):
        w = np.empty(E, dtype=np.float64)
        w[order[l]] = mass                       # Zipf mass per expert id
        free = np.ones((N, E), dtype=bool)
        for j in range(k):
            u_keep = g.random(N)
            u_draw = g.random(N)
            ww = np.where(free, w[None, :], 0.0)
            cum = np.cumsum(ww, axis=1)
            target = u_draw * cum[:, -1]
            drawn = np.minimum((cum <= target[:, None]).sum(axis=1), E - 1)
            # guard against landing on an exhausted id through rounding
            bad = ~free[rows, drawn]
            if bad.any():
                drawn[bad] = np.argmax(free[bad], axis=1)
            if l > 0:
                prev = routes[:, l - 1, j]
                use_prev = (u_keep < keep) & free[rows, prev]
                choice = np.where(use_prev, prev, drawn)
            else:
                choice = drawn
            routes[:, l, j] = choice
            free[rows, choice] = False
    return routes.astype(np.uint8)


def topic_routes(N, L, E, k, keep, s, topics, seed):
    """Predicted routes with topic structure, uint8 [N, L, k]: each token
    belongs to one of `topics` topics (uniformly, in random order along the
    token axis); a topic's tokens follow the Markov chain of predicted_routes
    over that topic's own expert popularity order (seed seed * 1009 + 1 + t),
    so tokens of one topic tend to share experts."""
    g = rng_for(seed, "misc")
    topic = g.integers(0, topics, size=N)
    routes = np.zeros((N, L, k), dtype=np.uint8)
    for t in range(topics):
        rows = np.flatnonzero(topic == t)
        if rows.size:
            routes[rows] = predicted_routes(rows.size, L, E, k, keep, s, seed * 1009 + 1 + t)
    return routes


def predicted_and_actual_routes(N, L, E, k, keep, s, acc, seed):
    """(actual, predicted) uint8 [N, L, k]: actual routes from the Markov chain
    of predicted_routes; the prediction keeps each choice with probability
    acc and otherwise names another expert the token does not use at that
    layer (a predictor of accuracy ~acc per choice)."""
    actual = predicted_routes(N, L, E, k, keep, s, seed)
    g = rng_for(seed, "misc")
    pred = actual.astype(np.int64).copy()
    for l in range(L):
        for j in range(k):
            flip = g.random(N) >= acc
            for i in np.nonzero(flip)[0]:
                used = set(actual[i, l].tolist()) | set(pred[i, l].tolist())
                free = [e for e in range(E) if e not in used]
                if free:
                    pred[i, l, j] = free[int(g.integers(len(free)))]
    return actual, pred.astype(np.uint8)


def route_boost_bias(routes, layer, E, boost, base=None):
    """Per-token bias [N, E] (f32): `boost` on the experts predicted for
    `layer`, plus an optional per-expert base bias."""
    routes = np.asarray(routes)
    N = routes.shape[0]
    b = np.zeros((N, E), dtype=np.float32)
    if base is not None:
        b += np.asarray(base, dtype=np.float32)[None, :]
    rows = np.repeat(np.arange(N), routes.shape[2])
    b[rows, routes[:, layer, :].reshape(-1).astype(np.int64)] += np.float32(boost)
    return b


def random_topk_idx(T, E, k, seed, skew=None):
    """k distinct expert ids per token, int32 [T, k] (inputs for the grouping
    step tested on its own). skew=None: uniform; else Zipf exponent."""
    g = rng_for(seed, "idx")
    if skew is None:
        keys = g.random((T, E))
    else:
        mass = np.arange(1, E + 1, dtype=np.float64) ** (-float(skew))
        keys = g.random((T, E)) ** (1.0 / mass[None, :])
    return np.argsort(-keys, axis=1)[:, :k].astype(np.int32)


def random_logits(T, E, seed, levels=None):
    """float32 [T, E] logits; levels=n quantises them to n values to force
    ties (including both signed zeros)."""
    g = rng_for(seed, "logits")
    z = g.standard_normal((T, E)).astype(np.float32)
    if levels is not None:
        z = (np.round(z * (levels / 4.0)) / (levels / 4.0)).astype(np.float32)
        negzero = (z == 0) & (g.random((T, E)) < 0.5)
        z[negzero] = np.float32(-0.0)
    return z
