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


def correction_slots(counts, slot_of_expert, S):
    """Host decision: the missed experts and the slots they are loaded into,
    in rounds when there are more misses than slots to take. counts [E] rows
    per expert, slot_of_expert [E] (-1 = not resident). Returns a list of
    (expert_ids, slot_ids) rounds."""
    counts = np.asarray(counts)
    slot = np.asarray(slot_of_expert)
    E = counts.shape[0]
    misses = [e for e in range(E) if counts[e] > 0 and slot[e] < 0]
    used = set(int(slot[e]) for e in range(E) if slot[e] >= 0 and counts[e] > 0)
    takeable = [s for s in range(S) if s not in used]
    if misses and not takeable:
        raise ValueError("every slot holds an expert the batch uses: no slot for the misses")
    rounds = []
    for i in range(0, len(misses), max(len(takeable), 1)):
        ex = misses[i:i + len(takeable)]
        rounds.append((np.array(ex, np.int32), np.array(takeable[:len(ex)], np.int32)))
    return rounds


def run_layer(x, topk_idx, topk_w, E, store, cache, slot_of_expert, token_ids=None, y=None,
              workspaces=None, copy_stream=None):
    """One MoE layer over the batch `token_ids` with the cache `cache` (device
    (w_gate, w_up, w_down) [S, ...]) holding the experts slot_of_expert maps
    (host int [E]), correcting misses from `store` (host tensors [E, ...]).
    Returns (y, info) with info = dict(misses, rounds, incomplete_before)."""
    torch = ops._torch()
    dev = x.device
    comp = torch.cuda.current_stream()
    copy = copy_stream if copy_stream is not None else torch.cuda.Stream(device=dev)
    n_tokens, k = topk_idx.shape
    T = token_ids.shape[0] if token_ids is not None else n_tokens
    H = x.shape[1]
    F = cache[0].shape[1]
    S = cache[0].shape[0]
    ws = workspaces or {}
    perm_ws = ws.get("permute")
    ffn_ws = ws.get("ffn")
    offs, rop, por, xp = ops.permute(x, topk_idx, E, token_ids=token_ids, workspace=perm_ws)
    slot_host = np.asarray(slot_of_expert, dtype=np.int32)
    slot_dev = torch.from_numpy(slot_host).to(dev)
    # resident experts first (compute stream)
    yp = torch.empty((T * k, H), dtype=x.dtype, device=dev)
    ops.expert_ffn(xp, offs, *cache, slot_of_expert=slot_dev, y_perm=yp, workspace=ffn_ws)
    # misses need the rows per expert on the host (one small copy)
    counts = torch.diff(offs).cpu().numpy()
    rounds = correction_slots(counts, slot_host, S)
    # the first round's loads go to slots the resident experts do not read, so
    # they run on the copy stream while the resident experts compute
    done = torch.cuda.Event()
    done.record(comp)
    y, inc = ops.combine(yp, topk_idx, topk_w, rop, token_ids=token_ids, slot_of_expert=slot_dev,
                         y=y)
    for r, (ex, sl) in enumerate(rounds):
        if r > 0:
            copy.wait_event(done)         # the previous round's slots are free again
        ops.load_experts(store, cache, ex, sl, stream=copy)
        loaded = torch.cuda.Event()
        loaded.record(copy)
        comp.wait_event(loaded)
        miss_slot = np.full(E, -1, np.int32)
        miss_slot[ex] = sl
        miss_dev = torch.from_numpy(miss_slot).to(dev)
        ops.expert_ffn(xp, offs, *cache, slot_of_expert=miss_dev, y_perm=yp, workspace=ffn_ws)
        ops.combine(yp, topk_idx, topk_w, rop, token_ids=token_ids, slot_of_expert=miss_dev, y=y,
                    accumulate=True, want_incomplete=False)
        done = torch.cuda.Event()
        done.record(comp)
    return y, {"misses": int(sum(len(ex) for ex, _ in rounds)), "rounds": len(rounds),
               "incomplete": inc}
