"""Pins of the KV-cache Merge/Reindex (Sec. 3.3.3) and of the residual layer
stack: identities of array indexing, the dense residual stack a one-expert
top-1 stack reduces to, and token independence."""
import numpy as np

import oracle
from paper_2410_17954_amd import synth


def test_round_bf16_against_bit_rounding_of_float32():
    # an independent rounding: float32 bit patterns, round half to even at bit 16
    x = np.random.default_rng(0).standard_normal(50000).astype(np.float32) * 7
    assert np.array_equal(oracle.round_bf16(x.astype(np.float64)),
                          synth.values(synth.bf16_bits(x)))
    # float64 values between bfloat16 neighbours: 1 + 2^-8 is a tie (to even, 1),
    # anything above it rounds up
    assert oracle.round_bf16(np.array([1 + 2.0 ** -8, 1 + 2.0 ** -8 + 2.0 ** -40,
                                       1 + 3 * 2.0 ** -8])).tolist() == [1.0, 1 + 2.0 ** -7,
                                                                          1 + 2.0 ** -6]


def test_merge_of_consecutive_slices_is_the_whole_cache():
    g = np.random.default_rng(1)
    whole = g.standard_normal((3, 29, 5))
    parts = [whole[:, :7], whole[:, 7:7], whole[:, 7:20], whole[:, 20:]]
    assert np.array_equal(oracle.kv_merge(parts), whole)


def test_gather_identity_and_inverse_permutation():
    g = np.random.default_rng(2)
    merged = g.standard_normal((2, 40, 3))
    perm = g.permutation(40)
    assert np.array_equal(oracle.kv_gather(merged, np.arange(40)), merged)
    inv = np.empty(40, dtype=np.int64)
    inv[perm] = np.arange(40)
    back = oracle.kv_gather(oracle.kv_gather(merged, perm), inv)
    assert np.array_equal(back, merged)
    # one row by hand
    assert np.array_equal(oracle.kv_gather(merged, perm)[1, 5], merged[1, perm[5]])


def test_reindex_finds_every_token_in_its_new_batch():
    routes = synth.predicted_routes(37, 3, 8, 2, 0.6, 1.0, seed=3).astype(np.int64)
    perm, off, _, _ = oracle.schedule_multi(routes, 8, 3)
    batch_of, pos_of = oracle.kv_reindex(perm, off)
    sizes = np.diff(off)
    for gtok in range(37):
        b = batch_of[gtok]
        assert 0 <= pos_of[gtok] < sizes[b]
        assert perm[off[b] + pos_of[gtok]] == gtok
    # the schedule's new batches read their KV rows through the merged cache
    g = np.random.default_rng(4)
    batches = [g.standard_normal((2, n, 4)) for n in (20, 17)]   # the original two batches
    merged = oracle.kv_merge(batches)
    new = oracle.kv_gather(merged, perm)
    t = perm[off[2]]                                             # first token of new batch 2
    src = batches[0][:, t] if t < 20 else batches[1][:, t - 20]
    assert np.array_equal(new[:, off[2]], src)


def _stack_inputs(L, T=9, seed=5, E=None):
    cfg = synth.workload("tiny_fp32")
    layers = []
    for l in range(L):
        inp = synth.layer_inputs(cfg, seed=seed + l, T=T, parts=("router", "experts"))
        d = {k: synth.values(v) for k, v in inp.items()}
        if E is not None:
            d = {"w_router": d["w_router"][:E], "w_gate": d["w_gate"][:E],
                 "w_up": d["w_up"][:E], "w_down": d["w_down"][:E]}
        layers.append(d)
    x = synth.values(synth.layer_inputs(cfg, seed=seed, T=T, parts=("x",))["x"])
    return cfg, oracle.round_bf16(x), layers       # the stack's state is bf16


def test_one_expert_top1_stack_is_the_dense_residual_stack():
    cfg, x, layers = _stack_inputs(3, E=1)
    h, states, ins, idx = oracle.moe_stack(x, layers, 1)
    ref = x.copy()
    for d in layers:                                # written out with numpy alone
        g = ref @ d["w_gate"][0].T
        u = ref @ d["w_up"][0].T
        a = g / (1 + np.exp(-g)) * u
        ref = oracle.round_bf16(ref + a @ d["w_down"][0].T)
    assert np.allclose(h, ref, rtol=0, atol=1e-12)
    assert (idx == 0).all() and np.array_equal(ins[0], x)


def test_zero_experts_leave_the_state_unchanged():
    cfg, x, layers = _stack_inputs(2)
    for d in layers:
        d["w_down"] = np.zeros_like(d["w_down"])
    h, _, _, _ = oracle.moe_stack(x, layers, cfg["k"], pre_norm=True)
    assert np.array_equal(h, x)


def test_tokens_are_independent_through_the_stack():
    cfg, x, layers = _stack_inputs(3, T=7)
    h, _, _, idx = oracle.moe_stack(x, layers, cfg["k"], pre_norm=True)
    for t in (0, 3, 6):
        ht, _, _, it = oracle.moe_stack(x[t:t + 1], layers, cfg["k"], pre_norm=True)
        assert np.allclose(ht[0], h[t], rtol=0, atol=1e-12)
        assert np.array_equal(it[:, 0], idx[:, t])


def test_stack_state_is_bf16_between_layers():
    cfg, x, layers = _stack_inputs(2)
    h, states, ins, _ = oracle.moe_stack(x, layers, cfg["k"], pre_norm=True)
    for a in (states[1], ins[0], ins[1], h):
        assert np.array_equal(oracle.round_bf16(a), a)


def test_rms_norm_closed_forms():
    g = np.random.default_rng(6)
    h = g.standard_normal((5, 64)) * 3
    r = oracle.rms_norm(h, eps=0.0)
    assert np.allclose((r * r).mean(axis=1), 1.0, rtol=1e-14)       # unit mean square
    assert np.allclose(oracle.rms_norm(7.5 * h, eps=0.0), r, rtol=1e-14)   # scale-free
    c = np.full((1, 16), -2.0)                                      # a constant row
    w = np.arange(16, dtype=np.float64)
    assert np.allclose(oracle.rms_norm(c, w, eps=0.25), -2.0 / np.sqrt(4.25) * w, rtol=1e-15)


def test_pre_norm_keeps_the_stack_bounded():
    # without the norm SwiGLU's growth compounds over layers; with it the
    # input of every block has unit mean square
    cfg, x, layers = _stack_inputs(4)
    _, _, ins, _ = oracle.moe_stack(x * 10, layers, cfg["k"], pre_norm=True)
    ms = (ins * ins).mean(axis=2)
    assert np.allclose(ms, 1.0, rtol=1e-2)
