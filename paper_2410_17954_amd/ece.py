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
