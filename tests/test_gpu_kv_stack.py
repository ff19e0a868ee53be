"""GPU parity of the KV-cache Merge/Reindex (Sec. 3.3.3) and of the residual
layer stack against the oracle. KV movement and index maps bit-exact; each
layer of the stack is checked from the state the GPU fed it (its h_trace), so
a one-ulp difference in an early layer cannot flip a later top-k decision:
top-k bit-exact, the next state within 1e-2 * max|y| + 2^-8 * |h + y| (the
layer's bf16 tolerance plus one bf16 rounding of the sum)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2410_17954_amd import ops, synth
from gpu_helpers import to_dev, to_host, vals

pytestmark = pytest.mark.gpu


def _bytes(shape, seed):
    return np.random.default_rng(seed).integers(0, 256, size=shape, dtype=np.uint8)


@pytest.mark.parametrize("row", [4096, 48, 6])
def test_merge_then_reindex_matches_the_oracle(row):
    L, sizes = 3, (700, 0, 513, 90)
    src = [_bytes((L, n, row), seed=n + row) for n in sizes]
    merged, err = ops.kv_gather([to_dev(s) for s in src])
    assert to_host(err)[0] == 0
    assert np.array_equal(to_host(merged), oracle.kv_merge(src))
    # the new layout from a B-way schedule of the unit's predicted routes
    N = sum(sizes)
    routes = synth.predicted_routes(N, 4, 16, 2, 0.6, 1.0, seed=row)
    perm, off, _, _ = ops.schedule_multi(to_dev(routes), 16, 3)
    new, err = ops.kv_gather([to_dev(s) for s in src], index=perm)
    assert to_host(err)[0] == 0
    ref = oracle.kv_gather(oracle.kv_merge(src), to_host(perm))
    assert np.array_equal(to_host(new), ref)
    b_of, p_of, err = ops.kv_reindex(perm, off)
    rb, rp = oracle.kv_reindex(to_host(perm), to_host(off))
    assert to_host(err)[0] == 0
    assert np.array_equal(to_host(b_of), rb) and np.array_equal(to_host(p_of), rp)


def test_gather_flags_out_of_range_ids_and_skips_their_rows():
    src = [_bytes((2, 10, 32), seed=1)]
    index = np.array([3, 10, 0, -1], dtype=np.int32)
    out = torch.full((2, 4, 32), 7, dtype=torch.uint8, device="cuda:0")
    out, err = ops.kv_gather([to_dev(s) for s in src], index=to_dev(index), out=out)
    o = to_host(out)
    assert to_host(err)[0] == 1
    assert np.array_equal(o[:, 0], src[0][:, 3]) and np.array_equal(o[:, 2], src[0][:, 0])
    assert (o[:, 1] == 7).all() and (o[:, 3] == 7).all()


def _layers(L, E, H, F, seed, S=None):
    g = np.random.default_rng(seed)
    S = E if S is None else S
    out = []
    for l in range(L):
        wr = synth.bf16_bits(g.standard_normal((E, H)).astype(np.float32) * np.float32(0.05))
        wg = synth.bf16_bits(g.standard_normal((S, F, H)).astype(np.float32) * np.float32(0.03))
        wu = synth.bf16_bits(g.standard_normal((S, F, H)).astype(np.float32) * np.float32(0.03))
        wd = synth.bf16_bits(g.standard_normal((S, H, F)).astype(np.float32) * np.float32(0.03))
        out.append((wr, wg, wu, wd))
    return out


def _check_layers(h_in, h_out_rows, trace, idx_trace, layers, k, slots=None, norms=None,
                  pre_norm=False, eps=1e-5):
    """Layer l from the GPU's own input trace[l][1] (its state trace[l][0]); the
    state after it is trace[l+1][0] (or the final rows)."""
    L = len(layers)
    for l in range(L):
        state = vals(trace[l][0])
        x = vals(trace[l][1])
        if pre_norm:            # the norm, within one bf16 step of the float64 value
            ref_x = oracle.rms_norm(state, None if norms is None else synth.values(norms[l]), eps)
            assert (np.abs(x - ref_x) <= 2.0 ** -7 * np.abs(ref_x) + 1e-6).all(), f"norm {l}"
        else:
            assert np.array_equal(x, state)
        wr, wg, wu, wd = (synth.values(a) for a in layers[l])
        ref = oracle.moe_layer(x, wr, k, wg, wu, wd,
                               slot_of_expert=None if slots is None else slots[l])
        assert np.array_equal(idx_trace[l], ref["idx"]), f"layer {l}: top-k"
        nxt = vals(trace[l + 1][0]) if l + 1 < L else h_out_rows
        want = state + ref["y"]
        tol = 1e-2 * np.abs(ref["y"]).max() + 2.0 ** -8 * np.abs(want)
        assert (np.abs(nxt - want) <= tol).all(), f"layer {l}: state"
    assert np.array_equal(vals(trace[0][0]), h_in)


@pytest.mark.parametrize("T,n,pre_norm,with_w", [(300, 300, False, False),
                                                 (257, 611, True, True),
                                                 (20, 64, True, False),
                                                 (129, 129, True, True)])
def test_stack_layer_by_layer(T, n, pre_norm, with_w):
    L, E, H, F, k = 3, 8, 256, 512, 2
    lay = _layers(L, E, H, F, seed=T)
    g = np.random.default_rng(n)
    h0 = synth.bf16_bits(g.standard_normal((n, H)).astype(np.float32) * np.float32(3))
    h = to_dev(h0)
    tok = None if T == n else np.sort(g.choice(n, size=T, replace=False)).astype(np.int32)
    norms = ([synth.bf16_bits((1 + 0.2 * g.standard_normal(H)).astype(np.float32))
              for _ in range(L)] if with_w else None)
    trace = torch.empty((L, 2, T, H), dtype=torch.bfloat16, device="cuda:0")
    itr = torch.empty((L, T, k), dtype=torch.int32, device="cuda:0")
    _, err = ops.stack_forward(h, [tuple(to_dev(a) for a in l_) for l_ in lay], k,
                               token_ids=None if tok is None else to_dev(tok),
                               pre_norm=pre_norm,
                               norm_weights=None if norms is None else [to_dev(w) for w in norms],
                               h_trace=trace, idx_trace=itr)
    torch.cuda.synchronize()
    assert to_host(err)[0] == 0
    rows = np.arange(n) if tok is None else tok
    hv = vals(h)
    _check_layers(synth.values(h0)[rows], hv[rows], trace, to_host(itr), lay, k, norms=norms,
                  pre_norm=pre_norm)
    rest = np.setdiff1d(np.arange(n), rows)
    assert np.array_equal(to_host(h)[rest], h0[rest])       # other rows untouched


def test_stack_with_a_resident_subset_per_layer():
    L, E, S, H, F, k, T = 2, 8, 5, 128, 256, 2, 200
    lay = _layers(L, E, H, F, seed=9, S=S)
    slots = np.full((L, E), -1, dtype=np.int32)
    slots[0, [0, 2, 3, 5, 7]] = [4, 0, 1, 2, 3]
    slots[1, [1, 2, 4, 6, 7]] = [0, 1, 2, 3, 4]
    g = np.random.default_rng(10)
    h0 = synth.bf16_bits(g.standard_normal((T, H)).astype(np.float32))
    h = to_dev(h0)
    trace = torch.empty((L, 2, T, H), dtype=torch.bfloat16, device="cuda:0")
    itr = torch.empty((L, T, k), dtype=torch.int32, device="cuda:0")
    ops.stack_forward(h, [tuple(to_dev(a) for a in l_) for l_ in lay], k,
                      slot_of_expert=to_dev(slots), S=S, h_trace=trace, idx_trace=itr)
    torch.cuda.synchronize()
    _check_layers(synth.values(h0), vals(h), trace, to_host(itr), lay, k, slots=slots)


def test_stack_full_shape_two_layers_sampled():
    """Mixtral-shaped pre-normalised blocks (H 4096, 8 experts of F 14336,
    top-2) over a 4096-token batch of an 8192-token unit; the oracle checks a
    seeded sample of tokens, layer by layer."""
    cfg = synth.workload("mixtral8x7b_layer")
    E, H, F, k = cfg["E"], cfg["H"], cfg["F"], cfg["k"]
    L, n, T = 2, 8192, 4096
    g = torch.Generator(device="cuda:0")
    g.manual_seed(11)
    dev = "cuda:0"
    lay = []
    for l in range(L):
        lay.append(tuple((torch.randn(s, device=dev, generator=g) * sc).to(torch.bfloat16)
                         for s, sc in (((E, H), 0.02), ((E, F, H), 0.02), ((E, F, H), 0.02),
                                       ((E, H, F), 0.02))))
    h = torch.randn((n, H), device=dev, generator=g).to(torch.bfloat16)
    h0 = to_host(h).copy()
    tok = torch.arange(1, n, 2, dtype=torch.int32, device=dev)          # the odd tokens
    trace = torch.empty((L, 2, T, H), dtype=torch.bfloat16, device=dev)
    itr = torch.empty((L, T, k), dtype=torch.int32, device=dev)
    ops.stack_forward(h, lay, k, token_ids=tok, pre_norm=True, h_trace=trace, idx_trace=itr)
    torch.cuda.synchronize()
    hv = vals(h)
    it = to_host(itr)
    sample = np.sort(np.random.default_rng(12).choice(T, size=20, replace=False))
    for l in range(L):
        state = vals(trace[l][0])[sample]
        x = vals(trace[l][1])[sample]
        ref_x = oracle.rms_norm(state)
        assert (np.abs(x - ref_x) <= 2.0 ** -7 * np.abs(ref_x) + 1e-6).all()
        wr, wg, wu, wd = (synth.values(to_host(a)) for a in lay[l])
        ref = oracle.moe_layer(x, wr, k, wg, wu, wd)
        assert np.array_equal(it[l][sample], ref["idx"])
        nxt = vals(trace[l + 1][0])[sample] if l + 1 < L else hv[1::2][sample]
        want = state + ref["y"]
        tol = 1e-2 * np.abs(ref["y"]).max() + 2.0 ** -8 * np.abs(want)
        assert (np.abs(nxt - want) <= tol).all()
    assert np.array_equal(to_host(h)[0::2], h0[0::2])


def test_stack_float32():
    # float32 state and weights: 16-byte rows of 4 values, the scalar norm path
    L, E, H, F, k, T = 2, 8, 128, 256, 2, 97
    g = np.random.default_rng(13)
    lay = [tuple(g.standard_normal(s).astype(np.float32) * np.float32(sc)
                 for s, sc in (((E, H), 0.05), ((E, F, H), 0.03), ((E, F, H), 0.03),
                               ((E, H, F), 0.03))) for _ in range(L)]
    h0 = g.standard_normal((T, H)).astype(np.float32)
    h = to_dev(h0)
    trace = torch.empty((L, 2, T, H), dtype=torch.float32, device="cuda:0")
    itr = torch.empty((L, T, k), dtype=torch.int32, device="cuda:0")
    ops.stack_forward(h, [tuple(to_dev(a) for a in l_) for l_ in lay], k, pre_norm=True,
                      h_trace=trace, idx_trace=itr)
    torch.cuda.synchronize()
    tr, it, hv = to_host(trace).astype(np.float64), to_host(itr), to_host(h).astype(np.float64)
    for l in range(L):
        state, x = tr[l][0], tr[l][1]
        assert np.allclose(x, oracle.rms_norm(state), rtol=1e-5, atol=1e-6)
        wr, wg, wu, wd = (a.astype(np.float64) for a in lay[l])
        ref = oracle.moe_layer(x, wr, k, wg, wu, wd)
        assert np.array_equal(it[l], ref["idx"])
        nxt = tr[l + 1][0] if l + 1 < L else hv
        assert np.abs(nxt - (state + ref["y"])).max() <= 1e-4 * np.abs(ref["y"]).max() + 1e-5
