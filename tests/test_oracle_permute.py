"""Pins of the expert-major grouping oracle."""
import numpy as np
import pytest

import oracle
from paper_2410_17954_amd import synth


def _check(x, idx, E, token_ids=None):
    off, rop, por, xp = oracle.permute(x, idx, E, token_ids)
    k = idx.shape[1]
    tok = np.arange(idx.shape[0]) if token_ids is None else np.asarray(token_ids)
    P = len(tok) * k
    ep = np.array([idx[tok[p // k], p % k] for p in range(P)], dtype=np.int64)
    # counts sum to T*k and offsets bracket each expert's rows
    assert off[0] == 0 and off[-1] == P
    assert np.array_equal(np.diff(off), np.bincount(ep, minlength=E))
    # bijection
    assert np.array_equal(np.sort(rop), np.arange(P))
    assert np.array_equal(por[rop], np.arange(P))
    assert np.array_equal(rop[por], np.arange(P))
    # each row lies in its expert's range, and rows of one expert follow pair order
    for e in range(E):
        rows = por[off[e]:off[e + 1]]
        assert (ep[rows] == e).all()
        assert (np.diff(rows) > 0).all()
    # a library stable sort by expert gives the same grouping
    assert np.array_equal(por, np.argsort(ep, kind="stable"))
    # row contents are exact copies
    for p in range(P):
        assert np.array_equal(xp[rop[p]], x[tok[p // k]])
    return off, rop, por, xp


@pytest.mark.parametrize("T,E,k", [(1, 1, 1), (37, 8, 2), (64, 60, 4), (50, 64, 6), (20, 5, 5)])
def test_permutation_invariants(T, E, k):
    idx = synth.random_topk_idx(T, E, k, seed=T + E)
    x = np.arange(T * 3, dtype=np.float64).reshape(T, 3)
    _check(x, idx, E)


def test_skewed_and_empty_experts():
    idx = synth.random_topk_idx(80, 64, 2, seed=4, skew=2.0)
    off, *_ = _check(np.arange(80.0)[:, None], idx, 64)
    assert (np.diff(off) == 0).any()


def test_all_tokens_on_one_expert():
    idx = np.zeros((30, 1), dtype=np.int32) + 3
    off, rop, por, _ = _check(np.arange(30.0)[:, None], idx, 8)
    assert off.tolist() == [0, 0, 0, 0, 30, 30, 30, 30, 30]
    assert np.array_equal(rop, np.arange(30))


def test_token_ids_select_and_order_the_batch():
    idx = synth.random_topk_idx(40, 8, 2, seed=9)
    x = np.arange(40 * 2, dtype=np.float64).reshape(40, 2)
    tok = np.array([39, 3, 17, 0, 22])
    _check(x, idx, 8, tok)
