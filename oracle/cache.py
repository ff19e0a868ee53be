"""Expert cache engine (Sec. 3.4): cross-layer slot planning from predicted
demand (PLEC, Sec. 3.4.1), its run-time behaviour with real-time correction of
mispredictions (Sec. 3.4.2), and the per-layer LRU cache it is compared
against (Sec. 1 and the evaluation's hit-ratio comparison).

TEST INFRASTRUCTURE: a plain, slow definition that the product harness is
checked against. Readings (the paper describes the policy in prose and one
worked example, Sec. 3.4.1):
  * load order: every (layer, expert) with predicted demand > 0, layers in
    execution order, within a layer larger predicted demand first, equal
    demand lower expert id first;
  * before the first layer the cache (`budget` slots) is filled in that order;
    when a layer has run, the slots its experts held are free and are refilled
    with the next items of the order that belong to later layers;
  * at a layer, an expert the batch actually uses is a hit if it is resident;
    a miss is loaded at once (correction) into a free slot, else over an
    expert of the same layer that the batch does not use (latest in load order
    first), else over the resident item of a later layer that is latest in
    load order (it goes back to the order and may be loaded again); with no
    slot to take the miss is served without caching it;
  * experts finish and free their slots per layer (the paper frees them per
    expert; hits are the same, only the timing of the refill differs).
"""


def plec_order(demand):
    """demand[l][e] (ints) -> list of (l, e) with demand > 0 in load order."""
    items = []
    for l in range(len(demand)):
        for e in range(len(demand[l])):
            if demand[l][e] > 0:
                items.append((l, -int(demand[l][e]), e))
    items.sort()
    return [(l, e) for (l, _, e) in items]


def plec_run(pred_demand, actual_demand, budget):
    """Simulate one batch through all layers. Returns a dict with the initial
    prefetch (list of (l, e)), per-layer hits and needed counts, the number of
    loads, and the experts resident when each layer started."""
    order = plec_order(pred_demand)
    pos = {item: i for i, item in enumerate(order)}
    pending = list(order)                 # not loaded yet, in load order
    resident = []                         # list of (l, e)
    loads = 0

    def fill(current):
        nonlocal loads
        kept = []
        for item in pending:
            if item[0] < current:
                continue                  # its layer has run: never needed
            if len(resident) < budget:
                resident.append(item)
                loads += 1
            else:
                kept.append(item)
        pending[:] = kept

    fill(0)
    prefetch = list(resident)
    L = len(actual_demand)
    hits, needed, start_sets = [], [], []
    for l in range(L):
        start_sets.append(sorted(e for (ll, e) in resident if ll == l))
        need = [e for e in range(len(actual_demand[l])) if actual_demand[l][e] > 0]
        h = 0
        for e in need:
            if (l, e) in resident:
                h += 1
                continue
            loads += 1                    # the correction load
            if len(resident) < budget:
                resident.append((l, e))
                continue
            unwanted = [it for it in resident if it[0] == l and it[1] not in need]
            later = [it for it in resident if it[0] > l]
            if unwanted:
                victim = max(unwanted, key=lambda it: pos.get(it, -1))
            elif later:
                victim = max(later, key=lambda it: pos[it])
                pending.append(victim)
                pending.sort(key=lambda it: pos[it])
            else:
                continue                  # served without caching
            resident.remove(victim)
            resident.append((l, e))
        hits.append(h)
        needed.append(len(need))
        resident[:] = [it for it in resident if it[0] != l]
        fill(l + 1)
    return {"prefetch": prefetch, "hits": hits, "needed": needed, "loads": loads,
            "start_sets": start_sets}


def lru_run(actual_demands, capacity):
    """Per-layer LRU caches of `capacity` experts each, kept across batches.
    actual_demands: [batch][l][e]; a layer's used experts are looked up in
    ascending id. Returns (hits, needed) summed over batches and layers."""
    hits = needed = 0
    caches = {}
    for dem in actual_demands:
        for l in range(len(dem)):
            cache = caches.setdefault(l, [])      # least recent first
            for e in range(len(dem[l])):
                if dem[l][e] <= 0:
                    continue
                needed += 1
                if e in cache:
                    hits += 1
                    cache.remove(e)
                    cache.append(e)
                elif capacity > 0:
                    cache.append(e)
                    if len(cache) > capacity:
                        cache.pop(0)
    return hits, needed
