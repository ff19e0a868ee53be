"""GPU parity of moe_expert_ffn against the oracle's SwiGLU experts."""
import numpy as np
import pytest
import torch

import oracle
from paper_2410_17954_amd import ops, synth
from gpu_helpers import to_dev, to_host, vals, rel_max_err

pytestmark = pytest.mark.gpu


def _weights(S, F, H, seed, dtype="bf16", std=0.02):
    g = np.random.default_rng(seed)
    ws = [g.standard_normal(s).astype(np.float32) * np.float32(std)
          for s in ((S, F, H), (S, F, H), (S, H, F))]
    return [synth.bf16_bits(w) for w in ws] if dtype == "bf16" else ws


def _rows(R, H, seed, dtype="bf16"):
    x = np.random.default_rng(seed + 1).standard_normal((R, H)).astype(np.float32)
    return synth.bf16_bits(x) if dtype == "bf16" else x


def _run(counts, H, F, slot, S, seed, dtype="bf16", tol=1e-2, extra_rows=0):
    counts = np.asarray(counts)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    R = int(offsets[-1]) + extra_rows
    x = _rows(max(R, 1), H, seed, dtype)
    wg, wu, wd = _weights(S, F, H, seed, dtype)
    sentinel = 3.0
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    y = torch.full((max(R, 1), H), sentinel, dtype=tdt, device="cuda:0")
    ops.expert_ffn(to_dev(x), to_dev(offsets), to_dev(wg), to_dev(wu), to_dev(wd),
                   slot_of_expert=None if slot is None else to_dev(np.asarray(slot, np.int32)),
                   y_perm=y)
    torch.cuda.synchronize()
    got = vals(y)
    sl = np.arange(len(counts)) if slot is None else np.asarray(slot)
    ref, computed = oracle.expert_ffn(synth.values(x)[:offsets[-1]], offsets, sl,
                                      synth.values(wg), synth.values(wu), synth.values(wd))
    if computed.any():
        assert rel_max_err(got[:offsets[-1]][computed], ref[computed]) <= tol
    assert (got[:offsets[-1]][~computed] == sentinel).all()
    assert (got[offsets[-1]:] == sentinel).all()
    return got, ref, computed


def test_tiny_fp32_config():
    cfg = synth.workload("tiny_fp32")
    counts = np.bincount(synth.random_topk_idx(64, 8, 2, 1).ravel(), minlength=8)
    _run(counts, cfg["H"], cfg["F"], None, 8, seed=1, dtype="f32", tol=1e-4)


@pytest.mark.parametrize("counts,H,F", [
    ([0, 300, 17, 513], 256, 512),        # ragged, several row tiles, an empty expert
    ([900, 2, 20, 30], 256, 512),          # large batch: its few-row experts take the large tiles
    ([1], 64, 64),                         # one row
    ([256, 256], 128, 192),                # exact tiles, F not a multiple of 64
    ([700, 3, 0, 1029, 64], 512, 1408),    # Qwen-like F
    ([300, 5, 260], 136, 200),             # H, F not multiples of 32: general path
    ([40, 300], 264, 96),                  # general path, K tail inside a 64-deep step
    ([263, 544, 300, 1025, 0, 287], 256, 512),   # small last row tiles (7, 32, 44, 1, 31 rows)
    ([257, 7, 288], 512, 1408),            # small last row tiles next to a lone 7-row expert
    ([356, 326, 320, 321, 128, 96, 288], 256, 512),  # last tiles of 100, 70, 64, 65 rows stay in place, 32 goes last
    ([1400, 300, 2100], 256, 512),         # experts of 6 and 9 full-cost row tiles
])
def test_bf16_ragged_groups(counts, H, F):
    _run(counts, H, F, None, len(counts), seed=sum(counts) + H)


@pytest.mark.parametrize("counts,H,F", [
    ([300, 40, 200], 4096, 4096),      # both GEMMs split their only, partial round along K (2 pieces)
    ([300, 40, 200], 1024, 8192),      # the down projection in 4 pieces
    ([9, 1100, 257, 31], 512, 4096),   # split down projection over ragged tiles of every size
    ([280, 530], 1024, 4096),          # the down projection's split round holds small last row tiles (24, 18 rows)
])
def test_bf16_split_k_tail(counts, H, F):
    # Fewer tiles than compute units: the last round is split into K-pieces
    # whose fp32 partials are summed in a fixed order, so a second call gives
    # identical bits.
    got, _, _ = _run(counts, H, F, None, len(counts), seed=sum(counts) + F)
    again, _, _ = _run(counts, H, F, None, len(counts), seed=sum(counts) + F)
    np.testing.assert_array_equal(got, again)


def test_bf16_resident_subset_and_slot_order():
    counts = [100, 200, 50, 300, 10, 0]
    slot = [2, -1, 0, -1, 1, 3]
    _run(counts, 256, 384, slot, 4, seed=21, extra_rows=33)


def test_bf16_nothing_resident():
    _run([10, 20], 64, 64, [-1, -1], 2, seed=22)


def test_shared_experts_as_one_dense_group():
    # two shared experts of width F concatenated along F == one expert of width 2F
    T, H, F = 333, 256, 256
    g = np.random.default_rng(5)
    x = synth.bf16_bits(g.standard_normal((T, H)).astype(np.float32))
    wg, wu, wd = _weights(1, 2 * F, H, seed=5)
    y = ops.expert_ffn(to_dev(x), to_dev(np.array([0, T], np.int32)), to_dev(wg), to_dev(wu),
                       to_dev(wd))
    xs, G, Uw, D = synth.values(x), synth.values(wg)[0], synth.values(wu)[0], synth.values(wd)[0]
    ref = sum(oracle.swiglu(xs, G[s * F:(s + 1) * F], Uw[s * F:(s + 1) * F], D[:, s * F:(s + 1) * F])
              for s in range(2))
    assert rel_max_err(vals(y), ref) <= 1e-2


@pytest.mark.parametrize("name", ["mixtral8x7b_layer", "qwen15_moe_layer"])
def test_full_shape_every_row(name):
    """Full expert shapes (Mixtral: 8192 rows of 4096 over F 14336; Qwen: 32768
    rows over 60 experts of F 1408): every row of y_perm against the oracle,
    which evaluates each expert's rows as one batch."""
    cfg = synth.workload(name)
    seed = cfg["seed"]
    E, H, F, k = cfg["E"], cfg["H"], cfg["F"], cfg["k"]
    T = cfg["T"]
    idx = synth.random_topk_idx(T, E, k, seed=seed, skew=cfg["zipf_bias"])
    counts = np.bincount(idx.ravel(), minlength=E)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    R = int(offsets[-1])
    inp = synth.layer_inputs(cfg, seed, T=R, parts=("x", "experts"))
    x = inp["x"]
    y = ops.expert_ffn(to_dev(x), to_dev(offsets), to_dev(inp["w_gate"]), to_dev(inp["w_up"]),
                       to_dev(inp["w_down"]))
    got = vals(y)
    ref = np.empty((R, H))
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi > lo:
            ref[lo:hi] = oracle.swiglu(synth.values(x[lo:hi]), synth.values(inp["w_gate"][e]),
                                       synth.values(inp["w_up"][e]),
                                       synth.values(inp["w_down"][e]))
    assert rel_max_err(got, ref) <= 1e-2


@pytest.mark.parametrize("counts,H,F", [
    ([1], 64, 64),                          # one row, one K batch
    ([1, 3, 16, 0, 17, 2], 512, 1408),      # few-row experts beside one with 17 rows
    ([16, 16, 16, 16], 256, 512),           # every expert at the few-row limit
    ([2, 7, 0, 5], 192, 320),               # K = 6 and 10 steps of 32: partial batches
    ([17, 32, 16, 33, 24], 256, 416),       # two-tile experts (17..32 rows) beside the others
    ([31, 1, 29], 160, 96),                 # K = 5 and 3 steps: every wave's range is short
    ([33, 48, 49, 64, 1, 17], 256, 416),    # three and four row tiles beside one and two
    ([65, 80, 96, 40, 3], 192, 320),        # five and six row tiles; K = 6 and 10 steps
    ([70, 2, 50], 160, 96),                 # down projection 160 wide: a half-empty last unit
    ([96, 96], 512, 1408),                  # every expert at the few-row limit (96 rows)
    ([81, 0, 0, 35], 128, 64),              # K = 4 and 2 steps with six and three row tiles
])
def test_bf16_few_rows_per_expert(counts, H, F):
    # in decode-sized batches experts with at most 96 rows take the
    # weight-streaming kernel
    _run(counts, H, F, None, len(counts), seed=sum(counts) + H + F)


@pytest.mark.parametrize("counts,slot,S,extra", [
    ([3, 0, 16, 1, 120, 9], [1, 0, -1, 3, 2, -1], 4, 5),
    ([97, 5, 60, 33], [2, 0, 1, -1], 3, 0),     # 97 rows: one row past the few-row limit
])
def test_bf16_few_rows_resident_subset(counts, slot, S, extra):
    # decode-sized batch (at most 64 rows per expert on average) with one
    # expert large enough for the large tiles
    _run(counts, 256, 384, slot, S, seed=23 + sum(counts), extra_rows=extra)


def test_bf16_few_rows_many_experts_subset():
    # decode-sized batch over 256 experts (the few-row list built from all of
    # them, ids sorted by row tiles), a fifth of them not resident, many empty,
    # one row past the few-row limit
    g = np.random.default_rng(5)
    E = 256
    counts = np.where(g.random(E) < 0.4, 0, g.integers(1, 80, size=E))
    counts[17] = 97
    slot = np.full(E, -1, np.int32)
    res = np.flatnonzero(g.random(E) < 0.8)
    slot[res] = np.arange(len(res), dtype=np.int32)
    assert counts.sum() <= 64 * E
    _run(counts, 64, 96, slot, len(res), seed=5, extra_rows=3)


def test_bf16_few_rows_nothing_to_do():
    # decode-sized batch whose experts are all empty or not resident: the
    # launches find no work and the output keeps its sentinel
    _run([0, 5, 0, 9], 128, 256, [0, -1, 1, -1], 2, seed=8, extra_rows=4)


@pytest.mark.parametrize("T,lo,hi", [(24, 1, 16), (100, 17, 32), (160, 33, 64), (256, 49, 96)])
def test_full_shape_decode_batch(T, lo, hi):
    """Decode-sized batch at the full 8-expert shape (H 4096, F 14336): 24,
    100, 160 or 256 tokens with top-2 give at most one, two, four or six
    16-row tiles per expert; every row is checked."""
    cfg = synth.workload("mixtral8x7b_layer")
    E, H, F, k = cfg["E"], cfg["H"], cfg["F"], cfg["k"]
    idx = synth.random_topk_idx(T, E, k, seed=77)
    counts = np.bincount(idx.ravel(), minlength=E)
    assert lo <= counts.max() <= hi
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    R = int(offsets[-1])
    inp = synth.layer_inputs(cfg, 2, T=R, parts=("x", "experts"))
    x = inp["x"]
    y = ops.expert_ffn(to_dev(x), to_dev(offsets), to_dev(inp["w_gate"]), to_dev(inp["w_up"]),
                       to_dev(inp["w_down"]))
    got = vals(y)
    ref = np.empty((R, H))
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi > lo:
            ref[lo:hi] = oracle.swiglu(synth.values(x[lo:hi]), synth.values(inp["w_gate"][e]),
                                       synth.values(inp["w_up"][e]), synth.values(inp["w_down"][e]))
    assert rel_max_err(got, ref) <= 1e-2


def test_bf16_many_experts_large_tiles():
    # 256 experts, a third of them empty and some non-resident, the rest from 1
    # to 700 rows: too many rows for the few-row kernels, so every tile's
    # expert is found among long flat stretches of the row-tile prefix
    g = np.random.default_rng(91)
    E = 256
    counts = np.where(g.random(E) < 0.35, 0, g.integers(1, 700, size=E))
    slot = np.full(E, -1, np.int32)
    res = np.flatnonzero(g.random(E) < 0.8)
    slot[res] = np.arange(len(res), dtype=np.int32)
    assert counts.sum() > 32 * E
    _run(counts, 64, 96, slot, len(res), seed=91)
