"""Pins of the routing-path-predictor forward (Sec. 3.2): T5's bucket formula
(by hand at its exact boundaries, by the real-valued formula elsewhere),
closed forms of attention and the blocks with parts of the weights zeroed,
causality of the decoder, independence of sequences, and the size reading."""
import math

import numpy as np
import pytest

from oracle import rpp

DIMS = dict(vocab=50, d_model=16, n_heads=4, d_ff=32, n_enc=2, n_dec=2, L=3, E=5,
            num_buckets=32, max_distance=128, eps=1e-6)


def _weights(dims, seed=0, scale=0.3):
    return np.random.default_rng(seed).standard_normal(rpp.n_weights(dims)) * scale


def _real_bucket(n, bidirectional, nb=32, D=128):
    """T5's formula in real arithmetic (used away from its exact boundaries)."""
    ret = 0
    if bidirectional:
        nb //= 2
        ret += nb if n < 0 else 0
        n = abs(n)
    else:
        n = max(n, 0)
    m = nb // 2
    if n < m:
        return ret + n
    large = m + int(math.log(n / m) / math.log(D / m) * (nb - m))
    return ret + min(large, nb - 1)


def test_buckets_by_hand_and_by_formula():
    # bidirectional: 8 + floor(2 log2(n/8)); exact boundaries at n = 16, 32, 64
    assert [rpp.bucket(n, True, 32, 128) for n in (0, 7, 8, 15, 16, 31, 32, 63, 64, 127, 128,
                                                   -1, -16, -500)] == \
        [0, 7, 8, 9, 10, 11, 12, 13, 14, 15, 15, 17, 26, 31]
    # causal: 16 + floor(16 log2(n/16) / 3); future keys clip to 0
    assert [rpp.bucket(n, False, 32, 128) for n in (-5, 0, 15, 16, 32, 64, 127, 128)] == \
        [0, 0, 15, 16, 21, 26, 31, 31]
    for n in range(-300, 300):
        for bi in (True, False):
            x = abs(n) if bi else max(n, 0)
            if x and math.log2(x) == int(math.log2(x)):
                continue                               # exact boundaries: by hand above
            assert rpp.bucket(n, bi, 32, 128) == _real_bucket(n, bi), (n, bi)


def test_size_reading_is_near_the_papers_7_21_MB():
    dims = dict(vocab=32000, d_model=32, n_heads=4, d_ff=2048, n_enc=3, n_dec=3, L=32, E=8,
                num_buckets=32, max_distance=128, eps=1e-6)
    n = rpp.n_weights(dims)
    assert n == 32000 * 32 + 2 * 32 * 4 + 3 * (64 + 4096 + 131072) + 3 * (96 + 8192 + 131072) \
        + 64 + 32 * 8 * 32
    assert abs(n * 4 / 1e6 - 7.21) < 0.25


def test_zero_query_key_weights_give_the_mean_of_values():
    B, S, d, h = 1, 5, 8, 2
    g = np.random.default_rng(1)
    x = g.standard_normal((B, S, d))
    wv, wo = g.standard_normal((d, d)), np.eye(d)
    zero = np.zeros((d, d))
    full = rpp._attention(x, x, zero, zero, wv, wo, h, np.zeros((h, S, S)))
    assert np.allclose(full, np.broadcast_to((x @ wv.T).mean(axis=1, keepdims=True), x.shape))
    causal = np.where(np.tril(np.ones((S, S))) > 0, 0.0, -np.inf)[None].repeat(h, 0)
    out = rpp._attention(x, x, zero, zero, wv, wo, h, causal)
    v = x @ wv.T
    for i in range(S):
        assert np.allclose(out[0, i], v[0, :i + 1].mean(axis=0))


def test_zero_heads_give_one_half():
    w = _weights(DIMS)
    p = rpp.unpack(w, DIMS)
    p["heads"][:] = 0.0
    probs, logits = rpp.rpp_forward(np.zeros((2, 4), dtype=np.int64), w, DIMS)
    assert (logits == 0).all() and (probs == 0.5).all()


def test_identity_blocks_reduce_to_the_normed_embedding():
    # every sub-block's output projection zeroed: y = rms_norm(emb[id]) * dec_ln
    w = _weights(DIMS, seed=2)
    p = rpp.unpack(w, DIMS)
    for lay in p["enc"] + p["dec"]:
        for key in ("o", "wo", "co"):
            if key in lay:
                lay[key][:] = 0.0
    ids = np.array([[3, 7, 7, 49]])
    _, logits = rpp.rpp_forward(ids, w, DIMS)
    e = p["emb"][ids]
    y = e / np.sqrt((e * e).mean(axis=-1, keepdims=True) + DIMS["eps"]) * p["dec_ln"]
    ref = (y @ p["heads"].T).reshape(1, 4, DIMS["L"], DIMS["E"])
    assert np.allclose(logits, ref, rtol=1e-12, atol=1e-12)


def test_decoder_is_causal_when_the_encoder_is_cut_off():
    w = _weights(DIMS, seed=3)
    p = rpp.unpack(w, DIMS)
    for lay in p["dec"]:
        lay["co"][:] = 0.0                              # no cross-attention output
    ids = np.array([[1, 2, 3, 4, 5, 6]])
    _, a = rpp.rpp_forward(ids, w, DIMS)
    ids2 = ids.copy()
    ids2[0, 4:] = [40, 41]
    _, b = rpp.rpp_forward(ids2, w, DIMS)
    assert np.array_equal(a[0, :4], b[0, :4]) and not np.allclose(a[0, 4:], b[0, 4:])


def test_sequences_are_independent_and_the_position_bias_is_used():
    w = _weights(DIMS, seed=4)
    ids = np.random.default_rng(5).integers(0, 50, size=(3, 7))
    _, all3 = rpp.rpp_forward(ids, w, DIMS)
    for b in range(3):
        _, one = rpp.rpp_forward(ids[b:b + 1], w, DIMS)
        assert np.allclose(one[0], all3[b], rtol=1e-12, atol=1e-12)
    # the relative-position bias tables take part: zeroing them changes the logits
    w0 = w.copy()
    p0 = rpp.unpack(w0, DIMS)
    p0["enc_rel"][:] = 0.0
    p0["dec_rel"][:] = 0.0
    _, nob = rpp.rpp_forward(ids, w0, DIMS)
    assert not np.allclose(nob, all3)


def _bias_only_attention(S, bidirectional, hot_bucket, beta):
    """One head whose scores come from the relative-position table alone (zero
    query and key weights), with a table that is beta on `hot_bucket` and zero
    elsewhere; the values are the one-hot rows of the identity, so row i of
    the output is query i's attention distribution over the keys."""
    h = 1
    rel = np.zeros((32, h))
    rel[hot_bucket, 0] = beta
    bias = rpp.position_bias(S, rel, bidirectional, 32, 128)
    x = np.eye(S)[None]                                # [1, S, S]: token j -> e_j
    zero = np.zeros((S, S))
    return rpp._attention(x, x, zero, zero, np.eye(S), np.eye(S), h, bias)[0]


def test_position_bias_direction_causal_by_hand():
    # Decoder (causal): query i sees keys j <= i at distance n = i - j >= 0.
    # The bucket of distance 1 (bucket 1) carries ln 3, every other bucket 0:
    #   query 0: only key 0                          -> [1, 0, 0]
    #   query 1: key 0 (n=1, weight 3), key 1 (n=0)  -> [3/4, 1/4, 0]
    #   query 2: keys 0 (n=2), 1 (n=1, weight 3), 2  -> [1/5, 3/5, 1/5]
    # With the distance taken the other way round (key - query) every visible
    # key would clip to bucket 0 and the table entry would never be read.
    p = _bias_only_attention(3, False, 1, math.log(3.0))
    np.testing.assert_allclose(p, [[1, 0, 0], [0.75, 0.25, 0], [0.2, 0.6, 0.2]], atol=1e-15)
    # bucket 0 (distance 0) differs from bucket 1: weighting it instead favours
    # the diagonal
    p0 = _bias_only_attention(3, False, 0, math.log(3.0))
    np.testing.assert_allclose(p0, [[1, 0, 0], [0.25, 0.75, 0], [0.2, 0.2, 0.6]], atol=1e-15)


def test_position_bias_direction_bidirectional_by_hand():
    # Encoder: keys before the query (n = i - j > 0) take the lower half of the
    # buckets, keys after it (n < 0) the upper half (16 + |n|). ln 3 on bucket
    # 1 (one step back):
    #   query 0: no key one step back                 -> uniform [1/3, 1/3, 1/3]
    #   query 1: key 0 weighted 3                      -> [3/5, 1/5, 1/5]
    #   query 2: key 1 weighted 3                      -> [1/5, 3/5, 1/5]
    p = _bias_only_attention(3, True, 1, math.log(3.0))
    np.testing.assert_allclose(p, [[1 / 3, 1 / 3, 1 / 3], [0.6, 0.2, 0.2], [0.2, 0.6, 0.2]],
                               atol=1e-15)
    # ln 3 on bucket 17 (one step ahead) mirrors it
    p = _bias_only_attention(3, True, 17, math.log(3.0))
    np.testing.assert_allclose(p, [[0.2, 0.6, 0.2], [0.2, 0.2, 0.6], [1 / 3, 1 / 3, 1 / 3]],
                               atol=1e-15)
