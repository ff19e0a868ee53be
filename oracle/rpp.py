"""Forward pass of the routing path predictor (RPP, Sec. 3.2): a T5-style
encoder-decoder over a batch of B sequences of S tokens whose L heads give,
for every token, logits over the E experts of each MoE layer; the activation
probabilities (B, S, L, E) are their sigmoids (the multi-label reading of the
predictor's binary cross-entropy training). Test infrastructure, written
plainly in float64.

Readings (the paper gives the family, hidden size 32 and feed-forward size
2048, Sec. 4.3.2, and nothing else):
  * T5 blocks: pre-norm RMS normalisation with a learned scale (eps 1e-6) and
    no mean subtraction; attention without the 1/sqrt(d_kv) factor and with a
    learned relative-position bias per head, shared by the layers of a stack;
    a ReLU feed-forward; no biases; the residual added after each sub-block;
    a final RMS norm on each stack's output.
  * The decoder reads the same token ids as the encoder (one pass, Fig. 2),
    with causal self-attention and cross-attention to the encoder output.
  * Heads: logits[l] = y W_l^T with W_l [E, d]; probabilities = sigmoid.
  * Relative-position buckets as T5's: distance n = query - key position;
    bidirectional (encoder) with half the buckets for each sign, causal
    (decoder) with n clipped at 0; the first half of a side's buckets are exact
    distances, the rest logarithmic up to max_distance. The logarithmic bucket
    m + floor((nb - m) * log(n / m) / log(D / m)) is evaluated exactly: for m
    and D powers of two it is m + floor((floor(log2(n ** a)) - a * log2(m)) / c)
    with a = nb - m and c = log2(D / m), where floor(log2(x)) of the integer
    x = n ** a is its bit length minus one.

Weights come as one float array in a fixed order (see `unpack`)."""
import numpy as np


def unpack(w, dims):
    """Views into the packed weight array, in this order (linear layers
    [out, in]):
      emb [V, d]; enc_rel [nb, h];
      per encoder layer: ln1 [d], q, k, v, o [d, d], ln2 [d], wi [dff, d], wo [d, dff];
      enc_ln [d]; dec_rel [nb, h];
      per decoder layer: ln1 [d], q, k, v, o [d, d], ln2 [d], cq, ck, cv, co [d, d],
                         ln3 [d], wi [dff, d], wo [d, dff];
      dec_ln [d]; heads [L*E, d]."""
    w = np.asarray(w, dtype=np.float64)
    V, d, h, dff = dims["vocab"], dims["d_model"], dims["n_heads"], dims["d_ff"]
    nb, L, E = dims["num_buckets"], dims["L"], dims["E"]
    pos = [0]

    def take(*shape):
        n = int(np.prod(shape))
        a = w[pos[0]:pos[0] + n].reshape(shape)
        pos[0] += n
        return a

    p = {"emb": take(V, d), "enc_rel": take(nb, h), "enc": [], "dec": []}
    for _ in range(dims["n_enc"]):
        p["enc"].append({"ln1": take(d), "q": take(d, d), "k": take(d, d), "v": take(d, d),
                         "o": take(d, d), "ln2": take(d), "wi": take(dff, d), "wo": take(d, dff)})
    p["enc_ln"] = take(d)
    p["dec_rel"] = take(nb, h)
    for _ in range(dims["n_dec"]):
        p["dec"].append({"ln1": take(d), "q": take(d, d), "k": take(d, d), "v": take(d, d),
                         "o": take(d, d), "ln2": take(d), "cq": take(d, d), "ck": take(d, d),
                         "cv": take(d, d), "co": take(d, d), "ln3": take(d), "wi": take(dff, d),
                         "wo": take(d, dff)})
    p["dec_ln"] = take(d)
    p["heads"] = take(L * E, d)
    if pos[0] != w.size:
        raise ValueError(f"weights hold {w.size} values, the dimensions need {pos[0]}")
    return p


def n_weights(dims):
    d, dff, h, nb = dims["d_model"], dims["d_ff"], dims["n_heads"], dims["num_buckets"]
    enc = 2 * d + 4 * d * d + 2 * d * dff
    dec = 3 * d + 8 * d * d + 2 * d * dff
    return (dims["vocab"] * d + 2 * nb * h + dims["n_enc"] * enc + dims["n_dec"] * dec + 2 * d
            + dims["L"] * dims["E"] * d)


def bucket(n, bidirectional, num_buckets, max_distance):
    """T5 relative-position bucket of distance n = query - key position, exact."""
    nb = num_buckets
    ret = 0
    if bidirectional:
        nb //= 2
        if n < 0:
            ret += nb
            n = -n
    else:
        n = max(n, 0)
    m = nb // 2
    if n < m:
        return ret + n
    if n >= max_distance:
        return ret + nb - 1
    a = nb - m
    c = (max_distance // m).bit_length() - 1           # log2(D / m)
    fl = (n ** a).bit_length() - 1                     # floor(log2(n ** a))
    j = (fl - a * (m.bit_length() - 1)) // c
    return ret + min(m + j, nb - 1)


def rms_norm(x, w, eps):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w


def _attention(xq, xkv, wq, wk, wv, wo, n_heads, bias):
    """xq [B, Sq, d], xkv [B, Sk, d]; bias [h, Sq, Sk] (or None); -inf masks."""
    B, Sq, d = xq.shape
    Sk = xkv.shape[1]
    dk = d // n_heads
    q = (xq @ wq.T).reshape(B, Sq, n_heads, dk).transpose(0, 2, 1, 3)
    k = (xkv @ wk.T).reshape(B, Sk, n_heads, dk).transpose(0, 2, 1, 3)
    v = (xkv @ wv.T).reshape(B, Sk, n_heads, dk).transpose(0, 2, 1, 3)
    s = q @ k.transpose(0, 1, 3, 2)                    # no 1/sqrt(dk): T5
    if bias is not None:
        s = s + bias[None]
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=-1, keepdims=True)
    o = (p @ v).transpose(0, 2, 1, 3).reshape(B, Sq, d)
    return o @ wo.T


def position_bias(S, rel, bidirectional, num_buckets, max_distance):
    """[h, S, S]: bias of query i and key j (causal: -inf above the diagonal)."""
    h = rel.shape[1]
    out = np.empty((h, S, S))
    for i in range(S):
        for j in range(S):
            if not bidirectional and j > i:
                out[:, i, j] = -np.inf
            else:
                out[:, i, j] = rel[bucket(i - j, bidirectional, num_buckets, max_distance)]
    return out


def rpp_forward(ids, weights, dims):
    """ids int [B, S]; returns (probs [B, S, L, E], logits [B, S, L, E])."""
    ids = np.asarray(ids, dtype=np.int64)
    B, S = ids.shape
    p = unpack(weights, dims)
    h, eps = dims["n_heads"], dims["eps"]
    nb, D = dims["num_buckets"], dims["max_distance"]
    enc_bias = position_bias(S, p["enc_rel"], True, nb, D)
    dec_bias = position_bias(S, p["dec_rel"], False, nb, D)
    x = p["emb"][ids]
    for lay in p["enc"]:
        x = x + _attention(rms_norm(x, lay["ln1"], eps), rms_norm(x, lay["ln1"], eps),
                           lay["q"], lay["k"], lay["v"], lay["o"], h, enc_bias)
        hid = np.maximum(rms_norm(x, lay["ln2"], eps) @ lay["wi"].T, 0.0)
        x = x + hid @ lay["wo"].T
    enc = rms_norm(x, p["enc_ln"], eps)
    y = p["emb"][ids]
    for lay in p["dec"]:
        n1 = rms_norm(y, lay["ln1"], eps)
        y = y + _attention(n1, n1, lay["q"], lay["k"], lay["v"], lay["o"], h, dec_bias)
        y = y + _attention(rms_norm(y, lay["ln2"], eps), enc, lay["cq"], lay["ck"], lay["cv"],
                           lay["co"], h, None)
        hid = np.maximum(rms_norm(y, lay["ln3"], eps) @ lay["wi"].T, 0.0)
        y = y + hid @ lay["wo"].T
    y = rms_norm(y, p["dec_ln"], eps)
    logits = (y @ p["heads"].T).reshape(B, S, dims["L"], dims["E"])
    return 1.0 / (1.0 + np.exp(-logits)), logits
