"""Pins of the expert-cache oracle (Sec. 3.4): the worked example of
Sec. 3.4.1, closed cases of the simulation, and hand-checked LRU sequences."""
import json
import os

import numpy as np

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_worked_example_of_plec():
    g = json.load(open(os.path.join(GOLDEN, "plec_worked_example.json")))
    r = oracle.plec_run(g["pred_demand"], g["pred_demand"], g["budget"])
    assert [list(it) for it in r["prefetch"]] == g["prefetch"]
    per_layer = [sum(1 for (l, _) in r["prefetch"] if l == ll) for ll in range(g["L"])]
    assert per_layer == g["initial_slots_per_layer"]
    assert r["start_sets"] == g["resident_when_layer_starts"]
    assert r["loads"] == g["loads"]
    assert r["hits"] == r["needed"] == [3, 2]


def test_load_order():
    d = [[0, 3, 3, 1], [5, 0, 0, 2]]
    assert oracle.plec_order(d) == [(0, 1), (0, 2), (0, 3), (1, 0), (1, 3)]


def test_perfect_prediction_with_room_for_every_layer_hits_everything():
    g = np.random.default_rng(3)
    for _ in range(50):
        L, E = g.integers(1, 6), g.integers(2, 12)
        d = (g.random((L, E)) < 0.4) * g.integers(1, 9, size=(L, E))
        budget = int((d > 0).sum(1).max())
        r = oracle.plec_run(d.tolist(), d.tolist(), budget)
        assert r["hits"] == r["needed"]
        assert r["loads"] == int((d > 0).sum())


def test_empty_cache_misses_everything():
    d = [[1, 0, 2], [0, 4, 0]]
    r = oracle.plec_run(d, d, 0)
    assert r["hits"] == [0, 0] and r["needed"] == [2, 1]
    assert r["prefetch"] == [] and r["loads"] == 3


def test_misprediction_is_corrected_over_an_unwanted_expert():
    # one slot; the prediction says expert 0, the batch uses expert 1
    r = oracle.plec_run([[1, 0]], [[0, 1]], 1)
    assert r["hits"] == [0] and r["needed"] == [1]
    assert r["loads"] == 2


def test_correction_evicts_the_latest_future_item_which_is_loaded_again():
    # two slots hold (0,0) and (1,0); layer 0 also needs expert 1: (1,0) is
    # evicted for it, and reloaded once layer 0 has run
    r = oracle.plec_run([[1, 0], [1, 0]], [[1, 1], [1, 0]], 2)
    assert r["hits"] == [1, 1]
    assert r["loads"] == 4


def test_lru_by_hand():
    # capacity 2: {0,1} cold misses, 2 evicts 0, 0 misses again, then 2 hits
    seq = [[[1, 1, 0]], [[0, 0, 1]], [[1, 0, 0]], [[0, 0, 1]]]
    assert oracle.lru_run(seq, 2) == (1, 5)
    # capacity >= E: only the first use of each expert misses
    assert oracle.lru_run(seq, 3) == (2, 5)
    assert oracle.lru_run(seq, 0) == (0, 5)
