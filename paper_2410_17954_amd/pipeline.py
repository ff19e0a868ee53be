"""Dual-batch inference pipeline (Sec. 3.3.4) over a stack of MoE layers.

Every two batches form a scheduling unit. For unit u the token scheduler
(Sec. 3.3.2) splits its 2T tokens into two new batches by predicted routing
path, the KV caches of the original batches are merged and reindexed into the
new layout (Sec. 3.3.3), and each new batch runs through the layer stack.
With `overlap` the planning of unit u+1 (routing prediction when it carries
token ids, token scheduler, KV merge/reindex)
runs on a second stream while unit u's layers run on the main stream; unit
u+1's layers wait for it through an event. Without it everything runs in
order on the main stream. Both orders give the same results bit for bit.
A plan's err word is set when the scheduler's result is not to be trusted or
a KV index is out of range; the caller checks it.

Routes come either with the unit (predicted elsewhere) or from the routing
path predictor (Sec. 3.2) run as part of the unit's plan, as in Fig. 1 and
Sec. 3.3.4, where the predictor and the token scheduler of the next unit run
beside the current one: the unit then carries token ids [B, S] (B*S tokens),
the predictor scores every expert of every layer for each token, and the k
highest per layer form its route (moe_route_binarize). Gating runs inside
each layer, on that layer's input.

Every step is a call of libmoeflow; this module only orders them on streams.
"""
from dataclasses import dataclass, field

from . import ops


@dataclass
class Unit:
    h: object                 # [N, H] hidden states, updated in place
    routes: object = None     # uint8 [N, L_pred, k] predicted routes, or None (predictor)
    kv: list = field(default_factory=list)   # caches of the original batches, [L_kv, T_b, ...]
    ids: object = None        # int32 [B, S] token ids (B*S = N) for the predictor


@dataclass
class UnitPlan:
    routes: object = None     # the routes the scheduler used (predicted here or given)
    perm: object = None
    offsets: object = None
    demand: object = None
    info: object = None
    kv_new: object = None
    batch_of: object = None
    pos_of: object = None
    err: object = None
    ready: object = None      # event: the plan is complete


class DualBatchPipeline:
    """Runs units through `layers` (list of (w_router, w_gate, w_up, w_down)
    device tensors per layer, every expert resident), each block RMS
    pre-normalised (norm_weights: one [H] tensor per layer, or None for unit
    weights) unless pre_norm is False. predictor: None, or dict(weights=
    float32 device tensor, dims=moe_rpp_dims fields with E equal to the
    stack's) for units that carry token ids instead of routes."""

    def __init__(self, layers, k, E, n_tokens, max_iters=10, keep_original_if_worse=True,
                 overlap=True, pre_norm=True, norm_weights=None, eps=1e-5, predictor=None):
        import torch
        self.torch = torch
        self.layers = layers
        self.k, self.E = k, E
        self.max_iters, self.keep = max_iters, keep_original_if_worse
        self.overlap = overlap
        self.pre_norm, self.norm_weights, self.eps = pre_norm, norm_weights, eps
        h_dim = layers[0][0].shape[1]
        F = layers[0][1].shape[1]
        dev = layers[0][0].device
        self.dev = dev
        self.main = torch.cuda.current_stream(dev)
        self.side = torch.cuda.Stream(dev) if overlap else self.main
        T = n_tokens - n_tokens // 2
        dt = ops._dtype_code(layers[0][0])
        self.stack_ws = ops.workspace_tensor(ops.stack_workspace(T, h_dim, F, E, k, dt), dev)
        self._sched_ws = {}
        self._rpp_ws = {}
        self.predictor = predictor
        if predictor is not None and predictor["dims"]["E"] != E:
            raise ValueError("the predictor's heads must score the stack's E experts")
        self.err = torch.zeros(1, dtype=torch.int32, device=dev)

    def _predict(self, ids, err):
        """Predictor forward and per-layer top-k on the current stream: uint8
        routes [B*S, L, k]."""
        pr = self.predictor
        dims = pr["dims"]
        B, S = ids.shape
        if (B, S) not in self._rpp_ws:
            self._rpp_ws[(B, S)] = ops.workspace_tensor(
                ops.load_library().moe_rpp_workspace(B, S, ops.ctypes.byref(ops.rpp_dims(dims))),
                self.dev)
        _, logits, _ = ops.rpp_forward(ids, pr["weights"], dims, err=err, want_logits=True,
                                       workspace=self._rpp_ws[(B, S)])
        routes = ops.route_binarize(logits, self.k)          # [B, S, L, k]
        return routes.view(B * S, dims["L"], self.k)

    def _plan(self, unit):
        """Routing prediction (when the unit carries token ids), token
        scheduler and KV merge/reindex for one unit on the side stream."""
        torch = self.torch
        p = UnitPlan()
        if unit.routes is None and (unit.ids is None or self.predictor is None):
            raise ValueError("a unit needs routes, or token ids and a predictor")
        if self.overlap:
            # the side stream reads these; the caching allocator must not hand
            # their memory out again before it has
            for t in (unit.routes, unit.ids):
                if t is not None:
                    t.record_stream(self.side)
            for kv in unit.kv:
                kv.record_stream(self.side)
        with torch.cuda.stream(self.side):
            p.err = torch.zeros(1, dtype=torch.int32, device=self.dev)
            p.routes = unit.routes if unit.routes is not None else self._predict(unit.ids, p.err)
            N, L_pred, k = p.routes.shape
            if N != unit.h.shape[0]:
                raise ValueError("the unit's routes or token ids do not cover its tokens")
            key = (N, L_pred, k)
            if key not in self._sched_ws:
                self._sched_ws[key] = ops.workspace_tensor(
                    ops.schedule_multi_workspace(N, L_pred, self.E, k, 2), self.dev)
            p.perm, p.offsets, p.demand, p.info = ops.schedule_multi(
                p.routes, self.E, 2, max_iters=self.max_iters,
                keep_original_if_worse=self.keep, workspace=self._sched_ws[key], err=p.err)
            if unit.kv:
                p.kv_new, _ = ops.kv_gather(unit.kv, index=p.perm, err=p.err)
            p.batch_of, p.pos_of, _ = ops.kv_reindex(p.perm, p.offsets, err=p.err)
            p.ready = torch.cuda.Event()
            p.ready.record(self.side)
        return p

    def _execute(self, unit, plan):
        """Both new batches of the unit through the layer stack (main stream)."""
        torch = self.torch
        self.main.wait_event(plan.ready)
        # the side stream allocated these tensors; the main stream uses them too
        for t in (plan.routes, plan.perm, plan.offsets, plan.demand, plan.info, plan.kv_new,
                  plan.batch_of, plan.pos_of, plan.err):
            if t is not None:
                t.record_stream(self.main)
        N = unit.h.shape[0]
        n1 = N // 2                  # the two-way split's boundary (fixed by N: no readback)
        with torch.cuda.stream(self.main):
            for lo, hi in ((0, n1), (n1, N)):
                if hi > lo:
                    ops.stack_forward(unit.h, self.layers, self.k, token_ids=plan.perm[lo:hi],
                                      pre_norm=self.pre_norm, norm_weights=self.norm_weights,
                                      eps=self.eps, err=self.err, workspace=self.stack_ws)

    def run(self, units):
        """Runs every unit; returns their plans (perm, demand, new KV, maps)."""
        plans = []
        if not units:
            return plans
        if self.overlap:
            # whatever the caller enqueued on the main stream before this call
            # (the units' routes, KV caches, hidden states) is complete before
            # the side stream reads it
            produced = self.torch.cuda.Event()
            produced.record(self.main)
            self.side.wait_event(produced)
        nxt = self._plan(units[0])
        for u, unit in enumerate(units):
            cur = nxt
            if u + 1 < len(units):
                if self.overlap:
                    nxt = self._plan(units[u + 1])    # runs beside unit u's layers
                    self._execute(unit, cur)
                else:
                    self._execute(unit, cur)
                    nxt = self._plan(units[u + 1])
            else:
                self._execute(unit, cur)
            plans.append(cur)
        return plans
