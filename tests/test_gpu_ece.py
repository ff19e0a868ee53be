"""GPU checks of the expert cache engine's run time (Sec. 3.4): whole experts
copied from pinned host memory into cache slots, and a layer whose cache
misses some of the experts its batch uses, corrected by loading them while
the resident experts compute, equals the all-resident layer of the oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2410_17954_amd import ece, ops, synth
from gpu_helpers import DEV, rel_max_err, to_dev, to_host, vals

pytestmark = pytest.mark.gpu


def _store(inp):
    def host(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).pin_memory()
    return tuple(host(inp[n]) for n in ("w_gate", "w_up", "w_down"))


def _cache(store, S):
    return tuple(torch.zeros((S,) + tuple(t.shape[1:]), dtype=torch.bfloat16, device=DEV)
                 for t in store)


def test_load_experts_copies_whole_experts():
    cfg = dict(synth.workload("mixtral8x7b_layer"), H=256, F=512)
    store = _store(synth.layer_inputs(cfg, 3, T=8, parts=("experts",)))
    cache = _cache(store, 3)
    ops.load_experts(store, cache, [5, 0, 7], [2, 0, 1])
    torch.cuda.synchronize()
    for t, c in zip(store, cache):
        for e, s in ((5, 2), (0, 0), (7, 1)):
            assert torch.equal(c[s].cpu(), t[e])


def test_load_experts_rejects_bad_ids():
    cfg = dict(synth.workload("mixtral8x7b_layer"), H=64, F=64)
    store = _store(synth.layer_inputs(cfg, 3, T=8, parts=("experts",)))
    cache = _cache(store, 2)
    for ex, sl in (([0, 1], [1, 1]), ([8], [0]), ([0], [2]), ([-1], [0])):
        with pytest.raises(ops.MoeError):
            ops.load_experts(store, cache, ex, sl)


@pytest.mark.parametrize("S,resident,rounds", [
    (8, [0, -1, 1, -1, 2, 3, -1, -1], 1),   # four spare slots take the four misses at once
    (3, [0, 1, -1, -1, -1, -1, -1, -1], 4),  # one spare slot, then the two resident slots once
                                             # the resident experts are done: rounds of 1, 2, 1, 2
])
def test_corrected_layer_equals_all_resident_layer(S, resident, rounds):
    cfg = dict(synth.workload("mixtral8x7b_layer"), T=512, H=512, F=1024)
    E, k = cfg["E"], cfg["k"]
    inp = synth.layer_inputs(cfg, 7)
    x_d = to_dev(inp["x"])
    idx, w, _ = ops.route(x_d, to_dev(inp["w_router"]), k)
    store = _store(inp)
    cache = _cache(store, S)
    resident = np.array(resident, np.int32)
    ex = [e for e in range(E) if resident[e] >= 0]
    ops.load_experts(store, cache, ex, resident[ex])
    y, info = ece.run_layer(x_d, idx, w, E, store, cache, resident)
    torch.cuda.synchronize()
    counts = np.bincount(idx.cpu().numpy().ravel(), minlength=E)
    assert info["misses"] == int(((resident < 0) & (counts > 0)).sum()) > 0
    assert info["rounds"] == rounds
    full = oracle.moe_layer(synth.values(inp["x"]), synth.values(inp["w_router"]), k,
                            synth.values(inp["w_gate"]), synth.values(inp["w_up"]),
                            synth.values(inp["w_down"]))
    # two roundings of y: the resident sum, then the corrected one
    assert rel_max_err(vals(y), full["y"]) <= 2e-2
    inc = info["incomplete"].cpu().numpy().astype(bool)
    assert np.array_equal(inc, (resident[full["idx"]] < 0).any(axis=1))


def _plec_stack_case(seed, L=4, T=64, H=256, F=512, E=8, k=2):
    g = np.random.default_rng(seed)
    bf = lambda shape, sc: synth.bf16_bits((g.standard_normal(shape) * sc).astype(np.float32))
    routers = [bf((E, H), 0.05) for _ in range(L)]
    wg, wu = bf((L, E, F, H), 0.03), bf((L, E, F, H), 0.03)
    wd = bf((L, E, H, F), 0.03)
    h0 = bf((T, H), 1.0)
    return routers, (wg, wu, wd), h0


@pytest.mark.parametrize("budget,overlap", [(12, False), (8, False), (20, True), (12, True)])
def test_plec_stack_executes_the_plan(budget, overlap):
    """A 4-layer stack whose experts live in pinned host memory and a device
    cache smaller than the 32 (layer, expert) pairs: the plan's prefetch,
    corrections of mispredicted experts and refills of freed slots really run
    (copies on a second stream), the per-layer hits, needed and the loads
    equal the oracle's simulation of the same policy on the same demands, and
    the output equals the all-resident stack (bit for bit with one expert
    launch per layer; within 1e-2 when the resident experts run while the
    corrections load)."""
    L, T, E, k = 4, 64, 8, 2
    routers, (wg, wu, wd), h0 = _plec_stack_case(7)
    # reference: every expert resident, the same kernels through the stack
    layers = [(to_dev(routers[l]), to_dev(wg[l]), to_dev(wu[l]), to_dev(wd[l])) for l in range(L)]
    h_ref = to_dev(h0)
    trace = torch.empty((L, T, k), dtype=torch.int32, device=DEV)
    ops.stack_forward(h_ref, layers, k, pre_norm=False, idx_trace=trace)
    torch.cuda.synchronize()
    actual = np.stack([np.bincount(to_host(trace)[l].ravel(), minlength=E) for l in range(L)])
    # prediction: the true demand with two experts per layer mispredicted
    g = np.random.default_rng(budget)
    pred = actual.copy()
    for l in range(L):
        used, unused = np.flatnonzero(actual[l] > 0), np.flatnonzero(actual[l] == 0)
        pred[l, g.choice(used, 2, replace=False)] = 0
        if unused.size:
            pred[l, g.choice(unused, 1)] = 5
    store = tuple(torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).pin_memory()
                  for a in (wg, wu, wd))
    cache = tuple(torch.zeros((budget,) + tuple(t.shape[2:]), dtype=torch.bfloat16, device=DEV)
                  for t in store)
    h = to_dev(h0)
    st = ece.run_plec_stack(h, [lay[0] for lay in layers], store, cache, pred, k, budget,
                            overlap_corrections=overlap)
    torch.cuda.synchronize()
    assert np.array_equal(st["demand"], actual)
    ref = oracle.plec_run(pred.tolist(), actual.tolist(), budget)
    assert st["hits"] == ref["hits"] and st["needed"] == ref["needed"]
    assert st["loads"] == ref["loads"]
    assert sum(st["hits"]) < sum(st["needed"])          # the mispredictions were corrected
    if overlap:
        assert rel_max_err(vals(h), vals(h_ref)) <= 1e-2
    else:
        assert np.array_equal(to_host(h), to_host(h_ref))
