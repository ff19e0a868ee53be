"""GPU parity of moe_permute: maps and gathered rows bit-exact."""
import numpy as np
import pytest
import torch

import oracle
from paper_2410_17954_amd import ops, synth
from gpu_helpers import to_dev, to_host, DEV

pytestmark = pytest.mark.gpu


def _run(n_tokens, E, k, H, seed, token_ids=None, skew=None, dtype="bf16", idx=None):
    if idx is None:
        idx = synth.random_topk_idx(n_tokens, E, k, seed, skew=skew)
    g = np.random.default_rng(seed)
    if dtype == "bf16":
        x = synth.bf16_bits(g.standard_normal((n_tokens, H)).astype(np.float32))
    else:
        x = g.standard_normal((n_tokens, H)).astype(np.float32)
    off, rop, por, xp = ops.permute(to_dev(x), to_dev(idx), E,
                                    token_ids=None if token_ids is None else to_dev(token_ids))
    r_off, r_rop, r_por, r_xp = oracle.permute(x, idx, E, token_ids)
    assert np.array_equal(to_host(off), r_off)
    assert np.array_equal(to_host(rop), r_rop)
    assert np.array_equal(to_host(por), r_por)
    assert np.array_equal(to_host(xp), r_xp)     # bit patterns


@pytest.mark.parametrize("n,E,k,H", [(1, 1, 1, 8), (37, 8, 2, 64), (5000, 60, 4, 128),
                                     (1500, 64, 6, 256), (700, 256, 8, 16), (33, 5, 5, 8)])
def test_maps_and_rows_exact(n, E, k, H):
    _run(n, E, k, H, seed=n + E)


def test_skewed_with_empty_experts():
    _run(3000, 64, 2, 64, seed=3, skew=2.5)


def test_all_pairs_on_one_expert():
    idx = np.full((4100, 1), 6, dtype=np.int32)
    _run(4100, 8, 1, 32, seed=4, idx=idx)


def test_token_id_subset_in_scheduled_order():
    g = np.random.default_rng(5)
    tok = g.permutation(6000)[:2500].astype(np.int32)
    _run(6000, 8, 2, 64, seed=5, token_ids=tok)


def test_float32_rows():
    _run(300, 8, 2, 132, seed=6, dtype="f32")


def test_mixtral_full_size():
    _run(4096, 8, 2, 4096, seed=2)


def test_maps_only_without_rows():
    idx = synth.random_topk_idx(999, 16, 3, 8)
    off, rop, por, xp = ops.permute(None, to_dev(idx), 16)
    r_off, r_rop, r_por, _ = oracle.permute(np.zeros((999, 1)), idx, 16)
    assert xp is None
    assert np.array_equal(to_host(off), r_off) and np.array_equal(to_host(rop), r_rop)
    assert np.array_equal(to_host(por), r_por)


def test_maps_only_many_chunks():
    # 800K pairs: chunks at the largest size (128 tokens x 8 choices), hundreds
    # of chunks per expert column scan, every expert id in use.
    idx = synth.random_topk_idx(100_000, 256, 8, 9)
    off, rop, por, _ = ops.permute(None, to_dev(idx), 256)
    r_off, r_rop, r_por, _ = oracle.permute(np.zeros((100_000, 1)), idx, 256)
    assert np.array_equal(to_host(off), r_off) and np.array_equal(to_host(rop), r_rop)
    assert np.array_equal(to_host(por), r_por)
