"""GPU parity of moe_combine against the oracle's weighted sum (Sec. 2.1)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2410_17954_amd import ops, synth
from gpu_helpers import to_dev, to_host, vals, rel_max_err

pytestmark = pytest.mark.gpu


def _inputs(n_tokens, T, E, k, H, seed, dtype="bf16"):
    g = np.random.default_rng(seed)
    idx = synth.random_topk_idx(n_tokens, E, k, seed)
    w = g.random((n_tokens, k)).astype(np.float32)
    P = T * k
    rop = g.permutation(P).astype(np.int32)
    yp = g.standard_normal((P, H)).astype(np.float32)
    ys = g.standard_normal((T, H)).astype(np.float32)
    y0 = g.standard_normal((n_tokens, H)).astype(np.float32)
    if dtype == "bf16":
        yp, ys, y0 = synth.bf16_bits(yp), synth.bf16_bits(ys), synth.bf16_bits(y0)
    return idx, w, rop, yp, ys, y0


def _elementwise_ok(got, ref, k, w):
    # one bf16 rounding of a float32 sum of k + 2 terms
    scale = np.max(np.abs(ref))
    tol = 2.0 ** -8 * np.abs(ref) + 1e-5 * scale
    assert (np.abs(got - ref) <= tol).all()
    assert rel_max_err(got, ref) <= 1e-2


@pytest.mark.parametrize("T,E,k,H", [(1, 4, 1, 8), (77, 8, 2, 128), (2048, 64, 6, 256),
                                     (300, 64, 12, 64),      # k > 8: the general kernel
                                     (4096, 8, 2, 4096)])    # Mixtral batch
def test_all_resident(T, E, k, H):
    idx, w, rop, yp, _, _ = _inputs(T, T, E, k, H, seed=T)
    y, inc = ops.combine(to_dev(yp), to_dev(idx), to_dev(w), to_dev(rop))
    ref, rinc = oracle.combine(synth.values(yp), idx, w, rop)
    _elementwise_ok(vals(y), ref, k, w)
    assert np.array_equal(to_host(inc), rinc)


def test_misses_shared_and_token_subset():
    n, T, E, k, H = 500, 200, 16, 4, 64
    idx, w, rop, yp, ys, _ = _inputs(n, T, E, k, H, seed=11)
    tok = np.random.default_rng(1).permutation(n)[:T].astype(np.int32)
    slot = np.array([0, -1, 1, 2, -1, 3, 4, 5, -1, 6, 7, 8, 9, -1, 10, 11], dtype=np.int32)
    y0 = torch.full((n, H), 7.0, dtype=torch.bfloat16, device="cuda:0")
    y, inc = ops.combine(to_dev(yp), to_dev(idx), to_dev(w), to_dev(rop), token_ids=to_dev(tok),
                         slot_of_expert=to_dev(slot), y_shared=to_dev(ys), y=y0)
    ref, rinc = oracle.combine(synth.values(yp), idx, w, rop, tok, slot, synth.values(ys),
                               n_out=n, y_init=np.full((n, H), 0.0))
    got = vals(y)
    untouched = np.setdiff1d(np.arange(n), tok)
    assert (got[untouched] == 7.0).all()
    _elementwise_ok(got[tok], ref[tok], k, w)
    assert np.array_equal(to_host(inc), rinc)


def test_accumulate_adds_to_existing_output():
    n, E, k, H = 300, 8, 2, 64
    idx, w, rop, yp, _, y0 = _inputs(n, n, E, k, H, seed=12)
    y = to_dev(y0)
    ops.combine(to_dev(yp), to_dev(idx), to_dev(w), to_dev(rop), y=y, accumulate=True)
    ref, _ = oracle.combine(synth.values(yp), idx, w, rop, y_init=synth.values(y0))
    _elementwise_ok(vals(y), ref, k, w)


def test_float32():
    n, E, k, H = 64, 8, 2, 132
    idx, w, rop, yp, ys, _ = _inputs(n, n, E, k, H, seed=13, dtype="f32")
    y, _ = ops.combine(to_dev(yp), to_dev(idx), to_dev(w), to_dev(rop), y_shared=to_dev(ys))
    ref, _ = oracle.combine(yp, idx, w, rop, y_shared=ys)
    assert np.max(np.abs(to_host(y) - ref)) <= 1e-5 * np.max(np.abs(ref))
