"""Expert cache engine at run time for one MoE layer (Sec. 3.4).

The layer's cache holds S expert slots on the device; the full expert store
lives in host memory (pinned, so copies run asynchronously). After the
grouping, the experts the batch really uses but the cache does not hold are
the misses (the prediction that chose the resident set was wrong). Their
weights are copied on a second stream into slots that the resident
computation does not read -- free slots, or slots of resident experts that
the batch does not use -- while the resident experts compute (real-time
correction, Sec. 3.4.2); then the missed rows are computed and added into y
(moe_combine with accumulate). Every step is a library call; this module only
orders them on the two streams.
"""
import numpy as np

from . import ops


def correction_plan(counts, slot_of_expert, S):
    """Host decision: which missed experts are loaded into which slots, in
    rounds. counts [E] rows per expert, slot_of_expert [E] (-1 = not
    resident). Two groups of slots take misses: group 0, the slots the
    resident computation does not read (free, or holding a resident expert
    the batch does not use), usable at once; group 1, the slots of resident
    experts the batch uses, usable once the resident experts have been
    computed. Rounds alternate between the groups, so each round's loads wait
    only for the computation that last read its slots. Returns a list of
    (group, expert_ids, slot_ids)."""
    counts = np.asarray(counts)
    slot = np.asarray(slot_of_expert)
    E = counts.shape[0]
    misses = [e for e in range(E) if counts[e] > 0 and slot[e] < 0]
    busy = sorted(set(int(slot[e]) for e in range(E) if slot[e] >= 0 and counts[e] > 0))
    groups = [[s for s in range(S) if s not in set(busy)], busy]
    if misses and not any(groups):
        raise ValueError("no cache slot to load the missed experts into")
    rounds = []
    i, g = 0, 0 if groups[0] else 1
    while i < len(misses):
        sl = groups[g]
        if sl:
            ex = misses[i:i + len(sl)]
            rounds.append((g, np.array(ex, np.int32), np.array(sl[:len(ex)], np.int32)))
            i += len(ex)
        g = 1 - g
    return rounds


def run_layer(x, topk_idx, topk_w, E, store, cache, slot_of_expert, token_ids=None, y=None,
              workspaces=None, copy_stream=None):
    """One MoE layer over the batch `token_ids` with the cache `cache` (device
    (w_gate, w_up, w_down) [S, ...]) holding the experts slot_of_expert maps
    (host int [E]), correcting misses from `store` (host tensors [E, ...],
    pinned for the loads to overlap). The loads overwrite cache slots: on
    return the cache holds what the last rounds loaded. Returns (y, info)
    with info = dict(misses, rounds, incomplete) (incomplete: the tokens the
    resident experts alone did not complete)."""
    torch = ops._torch()
    dev = x.device
    comp = torch.cuda.current_stream()
    copy = copy_stream if copy_stream is not None else torch.cuda.Stream(device=dev)
    n_tokens, k = topk_idx.shape
    T = token_ids.shape[0] if token_ids is not None else n_tokens
    H = x.shape[1]
    S = cache[0].shape[0]
    ws = workspaces or {}
    offs, rop, por, xp = ops.permute(x, topk_idx, E, token_ids=token_ids,
                                     workspace=ws.get("permute"))
    # the misses need the rows per expert on the host: one small copy of the
    # offsets, differenced there
    counts = np.diff(offs.cpu().numpy().astype(np.int64))
    slot_host = np.asarray(slot_of_expert, dtype=np.int32)
    rounds = correction_plan(counts, slot_host, S)
    # every slot table goes up in one transfer, before any cross-stream wait
    tables = np.full((1 + len(rounds), E), -1, np.int32)
    tables[0] = slot_host
    for r, (_, ex, sl) in enumerate(rounds):
        tables[1 + r, ex] = sl
    tables_dev = torch.from_numpy(tables).pin_memory().to(dev, non_blocking=True)
    # resident experts (compute stream)
    yp = torch.empty((T * k, H), dtype=x.dtype, device=dev)
    ops.expert_ffn(xp, offs, *cache, slot_of_expert=tables_dev[0], y_perm=yp,
                   workspace=ws.get("ffn"))
    last_read = [None, torch.cuda.Event()]       # per slot group: its last reader
    last_read[1].record(comp)
    y, inc = ops.combine(yp, topk_idx, topk_w, rop, token_ids=token_ids,
                         slot_of_expert=tables_dev[0], y=y)
    for r, (g, ex, sl) in enumerate(rounds):
        if last_read[g] is not None:
            copy.wait_event(last_read[g])
        ops.load_experts(store, cache, ex, sl, stream=copy)
        loaded = torch.cuda.Event()
        loaded.record(copy)
        comp.wait_event(loaded)
        ops.expert_ffn(xp, offs, *cache, slot_of_expert=tables_dev[1 + r], y_perm=yp,
                       workspace=ws.get("ffn"))
        done = torch.cuda.Event()
        done.record(comp)
        last_read[g] = done
        ops.combine(yp, topk_idx, topk_w, rop, token_ids=token_ids,
                    slot_of_expert=tables_dev[1 + r], y=y, accumulate=True,
                    want_incomplete=False)
    return y, {"misses": int(sum(len(ex) for _, ex, _ in rounds)), "rounds": len(rounds),
               "incomplete": inc}


def run_plec_stack(h, routers, store, cache, pred_demand, k, budget, biases=None,
                   renormalize=True, copy_stream=None, overlap_corrections=False):
    """One batch through L residual MoE layers (x_l = h, h += MoE_l(x_l)) whose
    experts live in a host store and in a device cache of `budget` slots run
    by PLEC (Sec. 3.4.1) with real-time correction (Sec. 3.4.2), the policy of
    moe_plec_run executed step by step (ops.PlecPlanner):
      * before layer 0 the plan's prefetch is copied into the cache;
      * at layer l the batch is routed and grouped on the compute stream, the
        rows per expert come back to the host (one small copy: the layer's
        actual demand), the planner lists the correction loads, which the copy
        stream issues at once, and the layer's experts run with the slot table
        the planner gives, then combine adds their sum into h;
      * when layer l's experts have run, the slots they held are refilled with
        later layers' items in load order (the copy stream waits for them).
    Every copy that layer l's experts read is ordered before them by events.
    With overlap_corrections the experts that were already resident run
    while the corrections load, the corrected ones after (two expert
    launches into one y_perm); otherwise one launch after the loads.

    h [T, H] device, updated in place; routers: L device [E, H]; biases: None
    or L device float32 [T, E] (added to the router logits); store: (w_gate,
    w_up [L, E, F, H], w_down [L, E, H, F]) host tensors, pinned for the
    copies to overlap; cache: (w_gate, w_up [budget, F, H], w_down [budget,
    H, F]) device; pred_demand: host int [L, E] (tokens predicted per
    expert). budget >= E (every expert of one layer fits, so no miss is ever
    served without a slot). Returns dict(hits [L], needed [L], loads,
    bytes_loaded, demand [L, E] actual rows per expert)."""
    torch = ops._torch()
    dev = h.device
    comp = torch.cuda.current_stream()
    copy = copy_stream if copy_stream is not None else torch.cuda.Stream(device=dev)
    L = len(routers)
    E, H = routers[0].shape
    T = h.shape[0]
    if budget < E:
        raise ValueError("budget must hold every expert of one layer")
    if cache[0].shape[0] != budget:
        raise ValueError("the cache must have `budget` slots")
    planner = ops.PlecPlanner(np.asarray(pred_demand), budget)
    expert_bytes = sum(t[0, 0].numel() * t.element_size() for t in store)
    ready = {}                     # layer -> copy-stream event after its latest load
    stats = {"hits": [], "needed": [], "loads": 0, "bytes_loaded": 0,
             "demand": np.zeros((L, E), np.int64)}

    def issue(rows):
        """Copies listed (layer, expert, slot) rows on the copy stream."""
        if len(rows) == 0:
            return
        for l in sorted(set(int(r[0]) for r in rows)):
            sel = rows[rows[:, 0] == l]
            ops.load_experts(tuple(t[l] for t in store), cache, sel[:, 1], sel[:, 2],
                             stream=copy)
            stats["bytes_loaded"] += expert_bytes * len(sel)
            ev = torch.cuda.Event()
            ev.record(copy)
            ready[l] = ev
        stats["loads"] += len(rows)

    copy.wait_event(_recorded(torch, comp))   # the cache is free to overwrite
    issue(planner.prefetch)
    R = T * k
    idx = torch.empty((T, k), dtype=torch.int32, device=dev)
    gw = torch.empty((T, k), dtype=torch.float32, device=dev)
    yp = torch.empty((R, H), dtype=h.dtype, device=dev)
    ws_p = ops.workspace_tensor(ops.permute_workspace(T, k, E), dev)
    ws_f = ops.workspace_tensor(
        ops.expert_ffn_workspace(R, H, cache[0].shape[1], E, ops._dtype_code(h)), dev)
    for l in range(L):
        ops.route(h, routers[l], k, bias=None if biases is None else biases[l],
                  renormalize=renormalize, topk_idx=idx, topk_w=gw)
        offs, rop, _, xp = ops.permute(h, idx, E, workspace=ws_p)
        counts = np.diff(offs.cpu().numpy().astype(np.int64))
        stats["demand"][l] = counts
        slot, corr, hits, needed = planner.layer(l, counts)
        stats["hits"].append(hits)
        stats["needed"].append(needed)
        before = ready.get(l)
        issue(corr)
        slot_d = torch.from_numpy(slot).to(dev)
        if overlap_corrections and len(corr):
            early = slot.copy()
            early[corr[:, 1]] = -1                  # experts still loading
            late = np.full(E, -1, np.int32)
            late[corr[:, 1]] = slot[corr[:, 1]]
            if before is not None:
                comp.wait_event(before)
            ops.expert_ffn(xp, offs, *cache, slot_of_expert=torch.from_numpy(early).to(dev),
                           y_perm=yp, workspace=ws_f)
            comp.wait_event(ready[l])
            ops.expert_ffn(xp, offs, *cache, slot_of_expert=torch.from_numpy(late).to(dev),
                           y_perm=yp, workspace=ws_f)
        else:
            if l in ready:
                comp.wait_event(ready[l])
            ops.expert_ffn(xp, offs, *cache, slot_of_expert=slot_d, y_perm=yp, workspace=ws_f)
        done = _recorded(torch, comp)
        ops.combine(yp, idx, gw, rop, slot_of_expert=slot_d, y=h, accumulate=True,
                    want_incomplete=False)
        refill = planner.advance(l)
        if len(refill):
            copy.wait_event(done)                  # the freed slots were read by layer l
            issue(refill)
    comp.wait_stream(copy)
    return stats


def _recorded(torch, stream):
    ev = torch.cuda.Event()
    ev.record(stream)
    return ev
