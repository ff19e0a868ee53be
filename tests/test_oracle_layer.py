"""Pins of the composed layer: the textbook special cases a MoE layer reduces
to, and the resident-set rule."""
import itertools

import numpy as np
import pytest

import oracle
from paper_2410_17954_amd import synth


def _inputs(name="tiny_fp32", T=12, seed=1, parts=("x", "router", "experts", "shared", "bias")):
    cfg = synth.workload(name)
    inp = synth.layer_inputs(cfg, seed=seed, T=T, parts=parts)
    return cfg, {k: synth.values(v) for k, v in inp.items()}


def test_one_expert_top1_layer_is_the_dense_ffn():
    cfg, d = _inputs()
    wg, wu, wd = d["w_gate"][:1], d["w_up"][:1], d["w_down"][:1]
    for renorm in (True, False):
        out = oracle.moe_layer(d["x"], d["w_router"][:1], 1, wg, wu, wd, renormalize=renorm)
        assert np.allclose(out["y"], oracle.dense_ffn(d["x"], wg[0], wu[0], wd[0]),
                           rtol=1e-13, atol=1e-13)
        assert out["incomplete"].sum() == 0


def test_k_equals_E_is_the_soft_mixture():
    cfg, d = _inputs()
    E = cfg["E"]
    for renorm in (True, False):
        out = oracle.moe_layer(d["x"], d["w_router"], E, d["w_gate"], d["w_up"],
                               d["w_down"], renormalize=renorm)
        p = oracle.softmax(d["x"] @ d["w_router"].T)
        soft = sum(p[:, e:e + 1] * oracle.swiglu(d["x"], d["w_gate"][e], d["w_up"][e],
                                                 d["w_down"][e]) for e in range(E))
        assert np.allclose(out["y"], soft, rtol=1e-12, atol=1e-14)


def test_shared_experts_concatenate_along_F():
    cfg, d = _inputs("qwen15_moe_layer", T=5, parts=("x", "shared"))
    H, F, ns = cfg["H"], cfg["F"], cfg["n_shared"]
    wg, wu, wd = d["shared_gate"], d["shared_up"], d["shared_down"]
    x = d["x"]
    total = oracle.swiglu(x, wg, wu, wd)
    parts = sum(oracle.swiglu(x, wg[s * F:(s + 1) * F], wu[s * F:(s + 1) * F],
                              wd[:, s * F:(s + 1) * F]) for s in range(ns))
    assert np.allclose(total, parts, rtol=1e-12, atol=1e-14)


def test_token_permutation_equivariance():
    cfg, d = _inputs(T=10)
    args = (d["w_router"], cfg["k"], d["w_gate"], d["w_up"], d["w_down"])
    y = oracle.moe_layer(d["x"], *args)["y"]
    pi = np.random.default_rng(3).permutation(10)
    y2 = oracle.moe_layer(d["x"][pi], *args)["y"]
    assert np.allclose(y2, y[pi], rtol=1e-13, atol=1e-14)


def test_resident_plus_missed_equals_full_output():
    cfg, d = _inputs(T=16)
    E = cfg["E"]
    args = (d["w_router"], cfg["k"], d["w_gate"], d["w_up"], d["w_down"])
    full = oracle.moe_layer(d["x"], *args)
    resident = np.array([0, -1, 1, -1, 2, 3, -1, -1])
    # weights are indexed by slot: reorder them to match this slot table
    slot_w = lambda w: np.stack([w[e] for e in range(E) if resident[e] >= 0])
    part = oracle.moe_layer(d["x"], d["w_router"], cfg["k"], slot_w(d["w_gate"]),
                            slot_w(d["w_up"]), slot_w(d["w_down"]), slot_of_expert=resident)
    missed_slots = np.where(resident >= 0, -1, 0)
    missed_slots[missed_slots == 0] = np.arange((resident < 0).sum())
    miss_w = lambda w: np.stack([w[e] for e in range(E) if resident[e] < 0])
    z, idx, w = full["logits"], full["idx"], full["w"]
    yp, _ = oracle.expert_ffn(full["x_perm"], full["offsets"], missed_slots,
                              miss_w(d["w_gate"]), miss_w(d["w_up"]), miss_w(d["w_down"]))
    y2, _ = oracle.combine(np.nan_to_num(yp), idx, w, full["row_of_pair"],
                           slot_of_expert=missed_slots, y_init=part["y"])
    assert np.allclose(y2, full["y"], rtol=1e-12, atol=1e-14)
    flagged = (resident[idx] < 0).any(axis=1)
    assert np.array_equal(part["incomplete"].astype(bool), flagged)


def test_plan_slots_brute_force():
    g = np.random.default_rng(5)
    for trial in range(40):
        E = int(g.integers(1, 8))
        S = int(g.integers(0, E + 2))
        demand = g.integers(0, 4, size=E)
        slot = oracle.plan_slots(demand, S)
        n = min(S, E)
        best = None
        for sub in itertools.combinations(range(E), n):
            score = (-sum(demand[list(sub)]), sorted((-demand[e], e) for e in sub))
            if best is None or score < best[0]:
                best = (score, sub)
        chosen = [e for e in range(E) if slot[e] >= 0]
        assert sum(demand[chosen]) == -best[0][0]
        assert chosen == sorted(best[1])
        assert [slot[e] for e in chosen] == list(range(n))
