"""Per-layer resident set from predicted demand (the planning step of PLEC,
Sec. 3.4.1: the cache is filled with the experts the prediction says will be
used most, and experts outside the cache are misses at run time).

Reading: with S slots for a layer, the resident experts are the S with the
largest demand (equal demand: lower expert id first); they occupy slots
0..S-1 in ascending expert id. slot_of_expert[e] = -1 marks a non-resident
expert. Pinned in tests/test_oracle_layer.py by brute force over subsets.
"""
import numpy as np


def plan_slots(demand, S):
    """demand: int [E] -> slot_of_expert int64 [E]."""
    demand = np.asarray(demand, dtype=np.int64)
    E = demand.shape[0]
    S = max(0, min(int(S), E))
    order = np.lexsort((np.arange(E), -demand))
    chosen = np.sort(order[:S])
    slot = np.full(E, -1, dtype=np.int64)
    slot[chosen] = np.arange(S, dtype=np.int64)
    return slot
