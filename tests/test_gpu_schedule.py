"""GPU parity of moe_schedule against the oracle's token scheduler
(Sec. 3.3): perm, demand and info bit-exact."""
import json
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2410_17954_amd import ops, synth
from gpu_helpers import to_dev, to_host

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _check(routes, E, n1=None, max_iters=10, keep=True):
    routes = np.ascontiguousarray(routes, dtype=np.uint8)
    err = torch.zeros(1, dtype=torch.int32, device="cuda:0")
    perm, demand, info = ops.schedule(to_dev(routes), E, n1=n1, max_iters=max_iters,
                                      keep_original_if_worse=keep, err=err)
    rp, rd, ri = oracle.schedule(routes, E, n1, max_iters, keep)
    assert to_host(err)[0] == 0, "every grid barrier of the round loop completed"
    assert to_host(info).tolist() == ri.tolist()
    assert np.array_equal(to_host(perm), rp)
    assert np.array_equal(to_host(demand), rd)
    return ri


def test_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "ts_worked_example.json")))
    info = _check(np.array(g["routes"]), g["E"], g["n1"])
    assert info[5] == g["obj_optimum"]


@pytest.mark.parametrize("N,L,E,k,s", [(64, 4, 8, 2, 1.1), (1000, 8, 16, 2, 1.0),
                                       (777, 3, 64, 6, 1.0), (4097, 2, 256, 4, 0.5)])
def test_markov_routes(N, L, E, k, s):
    routes = synth.predicted_routes(N, L, E, k, 0.7, s, seed=N + L)
    _check(routes, E)


def test_route_grouped_mixtral_unit():
    cfg = synth.workload("mixtral8x7b_route_grouped")
    routes = synth.predicted_routes(cfg["T"], cfg["L"], cfg["E"], cfg["k"], cfg["keep"],
                                    cfg["zipf"], seed=3)
    info = _check(routes, cfg["E"])
    assert info[5] <= info[4]


def test_deepseek_unit_26_layers():
    cfg = synth.workload("deepseek_v2_lite_layer")
    routes = synth.predicted_routes(cfg["T"], cfg["L"], cfg["E"], cfg["k"], cfg["keep"],
                                    cfg["zipf"], seed=5)
    _check(routes, cfg["E"])


@pytest.mark.parametrize("n1", [0, 1, 5, 13])
def test_uneven_and_degenerate_splits(n1):
    routes = synth.predicted_routes(13, 3, 5, 2, 0.5, 0.8, seed=2)
    _check(routes, 5, n1=n1)


def test_single_token():
    _check(np.array([[[3, 1]]]), 4, n1=1)


def test_identical_routes():
    _check(np.tile(np.array([[2, 5], [1, 3], [0, 7]]), (300, 1, 1)), 8)


def test_planted_clusters():
    a = np.array([[0, 1]] * 6)
    b = np.array([[4, 5]] * 6)
    routes = np.stack([a] * 50 + [b] * 50)[np.random.default_rng(8).permutation(100)]
    info = _check(routes, 8)
    assert info[5] == 2 * 6 * 2


def test_iteration_limit_and_no_guard():
    routes = synth.predicted_routes(2000, 6, 8, 2, 0.5, 0.8, seed=9)
    _check(routes, 8, max_iters=1, keep=False)
    _check(routes, 8, max_iters=2, keep=False)


def test_k_equals_E():
    routes = np.tile(np.arange(4, dtype=np.uint8), (50, 2, 1))
    _check(routes, 4)


def test_first_word_ties_resolved_on_later_words():
    # With E = 64 the first path word is exactly layer 0: making layer 0 equal
    # for every token puts all of them in one run that the later words decide.
    routes = synth.predicted_routes(3000, 5, 64, 2, 0.7, 1.0, seed=31)
    routes[:, 0, :] = routes[0, 0, :]
    _check(routes, 64)


def test_repeated_multiword_paths():
    # 40 distinct paths of 3 words, each repeated many times: equal keys are
    # ordered by token index.
    base = synth.predicted_routes(40, 4, 40, 3, 0.5, 1.0, seed=32)
    pick = np.random.default_rng(33).integers(0, 40, size=2000)
    _check(base[pick], 40)


def test_several_positions_per_thread():
    # more tokens than 256 per compute unit: each thread of the round loop
    # owns several signature positions
    routes = synth.predicted_routes(70000, 3, 16, 2, 0.7, 1.0, seed=41)
    _check(routes, 16)


def test_long_paths_read_from_memory():
    # 32 layers x 256 experts = 128 words per path: the block's paths do not
    # fit in LDS next to the column counts and are read from memory
    routes = synth.predicted_routes(3000, 32, 256, 2, 0.7, 1.0, seed=42)
    _check(routes, 256)


# ----------------------------------------------------------------- B batches
def _check_multi(routes, E, B, max_iters=10, keep=True):
    routes = np.ascontiguousarray(routes, dtype=np.uint8)
    err = torch.zeros(1, dtype=torch.int32, device="cuda:0")
    perm, off, demand, info = ops.schedule_multi(to_dev(routes), E, B, max_iters=max_iters,
                                                 keep_original_if_worse=keep, err=err)
    rp, ro, rd, ri = oracle.schedule_multi(routes, E, B, max_iters, keep)
    assert to_host(err)[0] == 0
    assert to_host(off).tolist() == ro.tolist()
    if B > 1:
        assert to_host(info).tolist() == ri.tolist()
    assert np.array_equal(to_host(perm), rp)
    assert np.array_equal(to_host(demand), rd)
    return rp, ro, ri


@pytest.mark.parametrize("N,L,E,k,B,s", [(64, 4, 8, 2, 4, 1.1), (1000, 8, 16, 2, 3, 1.0),
                                         (777, 3, 64, 6, 5, 1.0), (4097, 2, 256, 4, 8, 0.5)])
def test_multi_way_markov_routes(N, L, E, k, B, s):
    routes = synth.predicted_routes(N, L, E, k, 0.7, s, seed=N + B)
    _check_multi(routes, E, B)


@pytest.mark.parametrize("B", [1, 2])
def test_multi_way_reductions(B):
    routes = synth.predicted_routes(301, 5, 8, 2, 0.6, 1.0, seed=51)
    _check_multi(routes, 8, B)


def test_multi_way_more_batches_than_tokens():
    routes = synth.predicted_routes(3, 2, 4, 2, 0.5, 0.8, seed=44)
    _check_multi(routes, 4, 8)


def test_multi_way_no_guard_and_one_round():
    routes = synth.predicted_routes(2000, 6, 8, 2, 0.5, 0.8, seed=52)
    _check_multi(routes, 8, 4, max_iters=1, keep=False)


def test_multi_way_mixtral_unit_four_batches():
    cfg = synth.workload("mixtral8x7b_layer")
    routes = synth.predicted_routes(2 * cfg["T"], cfg["L"], cfg["E"], cfg["k"], cfg["keep"],
                                    cfg["zipf"], seed=53)
    rp, ro, ri = _check_multi(routes, cfg["E"], 4)
    assert ro.tolist() == [0, 2048, 4096, 6144, 8192]


def test_multi_way_demand_too_large_for_lds():
    # 70 layers x 256 experts: the per-batch demand counts go straight to memory
    routes = synth.predicted_routes(300, 70, 256, 2, 0.7, 1.0, seed=54)
    _check_multi(routes, 256, 3)


def test_multi_way_many_small_nodes_per_level():
    # 200 batches of 15 tokens: the deepest levels hold more than 64 nodes,
    # each level's small nodes run as several launches of one block per node
    routes = synth.predicted_routes(3000, 4, 16, 2, 0.7, 1.0, seed=55)
    _check_multi(routes, 16, 200)


def test_multi_way_level_mixing_small_and_large_nodes():
    # 2300 tokens into 5 batches: the first level holds a 920-token node (one
    # block) beside a 1380-token node (general path); rows of 16 bytes
    routes = synth.predicted_routes(2300, 8, 64, 2, 0.7, 1.0, seed=56)
    _check_multi(routes, 64, 5)


def test_unaligned_routes():
    # routes starting one byte past an aligned address: byte loads throughout
    import torch
    N, L, E, k = 300, 8, 64, 2
    routes = np.ascontiguousarray(synth.predicted_routes(N, L, E, k, 0.7, 1.0, seed=57),
                                  dtype=np.uint8)
    buf = torch.empty(N * L * k + 1, dtype=torch.uint8, device="cuda:0")
    rt = buf[1:].view(N, L, k)
    rt.copy_(torch.from_numpy(routes))
    assert rt.data_ptr() % 16 != 0
    perm, demand, info = ops.schedule(rt, E)
    rp, rd, ri = oracle.schedule(routes, E)
    assert to_host(info).tolist() == ri.tolist()
    assert np.array_equal(to_host(perm), rp)
    assert np.array_equal(to_host(demand), rd)
    perm, off, demand, info = ops.schedule_multi(rt, E, 6)
    rp, ro, rd, ri = oracle.schedule_multi(routes, E, 6)
    assert to_host(info).tolist() == ri.tolist()
    assert np.array_equal(to_host(perm), rp)
    assert np.array_equal(to_host(demand), rd)


def test_two_way_million_tokens_properties():
    # 2^20 Mixtral-shaped tokens, beyond the oracle's reach: check what holds at
    # any size. perm is batch 1 then batch 2, each ascending; demand is the
    # batches' column counts; Eq. 2 before and after match them; the split is
    # the balanced threshold of delta = d(i, m1) - d(i, m2); after convergence
    # each medoid attains its batch's least distance sum.
    N, L, E, k = 1 << 20, 32, 8, 2
    base = synth.predicted_routes(1 << 17, L, E, k, 0.7, 1.1, seed=58)
    pick = np.random.default_rng(59).permutation(N) % base.shape[0]
    routes = np.ascontiguousarray(base[pick], dtype=np.uint8)
    n1 = N // 2
    perm, demand, info = ops.schedule(to_dev(routes), E, n1=n1)
    perm, demand, info = to_host(perm), to_host(demand), to_host(info)
    iters, conv, m1, m2, ob, oa, used, n1_out = (int(v) for v in info)
    assert n1_out == n1 and 1 <= iters <= 10 and conv in (0, 1)
    assert np.array_equal(np.sort(perm), np.arange(N))
    b1, b2 = perm[:n1], perm[n1:]
    assert np.all(np.diff(b1) > 0) and np.all(np.diff(b2) > 0)
    cols = (np.arange(L)[None, :, None] * E + routes.astype(np.int64)).reshape(N, L * k)

    def counts(tokens):
        return np.bincount(cols[tokens].ravel(), minlength=L * E)

    c1, c2 = counts(b1), counts(b2)
    assert np.array_equal(demand.reshape(2, -1), np.stack([c1, c2]))
    assert oa == int((c1 > 0).sum() + (c2 > 0).sum())
    o1, o2 = counts(np.arange(n1)), counts(np.arange(n1, N))
    assert ob == int((o1 > 0).sum() + (o2 > 0).sum())
    assert oa <= ob
    if used:
        assert np.array_equal(perm, np.arange(N)) and oa == ob
        return
    # packed paths as 0/1 rows; Hamming distances to the two medoids
    bits = np.zeros((N, L * E), dtype=np.uint8)
    np.put_along_axis(bits, cols, 1, axis=1)
    assert 0 <= m1 < N and 0 <= m2 < N
    d1 = (bits != bits[m1]).sum(axis=1, dtype=np.int64)
    d2 = (bits != bits[m2]).sum(axis=1, dtype=np.int64)
    delta = d1 - d2
    assert delta[b1].max() <= delta[b2].min()
    if conv:
        ones = bits.sum(axis=1, dtype=np.int64)
        for members, cnt, m in ((b1, c1, m1), (b2, c2, m2)):
            s = len(members) * ones[members] + ones[members].sum() \
                - 2 * cnt[cols[members]].sum(axis=1)
            assert m in set(members[s == s.min()].tolist())


def test_merge_passes_and_eight_positions_per_thread():
    # 300000 tokens: the signature order comes from merge passes over the
    # sorted 512-token chunks (586 chunks), and the round loop holds eight
    # positions per thread
    routes = synth.predicted_routes(300000, 3, 16, 2, 0.7, 1.0, seed=60)
    _check(routes, 16)


def test_sixteen_positions_per_thread():
    routes = synth.predicted_routes(600000, 3, 16, 2, 0.7, 1.0, seed=61)
    _check(routes, 16)


def test_merge_passes_with_ties_on_later_words():
    # 140000 tokens drawn from 3000 paths of 4 words each: the merges meet
    # equal first three words and decide on the fourth, then on the index
    base = synth.predicted_routes(3000, 2, 128, 2, 0.7, 1.0, seed=62)
    pick = np.random.default_rng(63).integers(0, 3000, size=140000)
    _check(base[pick], 128)
