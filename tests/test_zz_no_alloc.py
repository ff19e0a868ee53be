"""moe_permute_noalloc (static scratch, no allocation) against moe_permute:
identical maps and rows on two calls in a row, the second smaller, so the
second reuses the scratch the first left behind."""
import numpy as np
import pytest
import torch

from paper_2410_17954_amd import ops, synth
from gpu_helpers import to_dev, to_host

pytestmark = pytest.mark.gpu


def _pair(x_d, idx_d, E, tok_d, T):
    k = idx_d.shape[1]
    ref = ops.permute(x_d, idx_d, E, token_ids=tok_d, T=T)
    dev = idx_d.device
    outs = (torch.full((E + 1,), -7, dtype=torch.int32, device=dev),
            torch.full((T * k,), -7, dtype=torch.int32, device=dev),
            torch.full((T * k,), -7, dtype=torch.int32, device=dev),
            None if x_d is None else torch.zeros((T * k, x_d.shape[1]), dtype=x_d.dtype,
                                                 device=dev))
    got = ops.permute_noalloc(x_d, idx_d, E, *outs[:3], x_perm=outs[3], token_ids=tok_d, T=T)
    torch.cuda.synchronize()
    for a, b in zip(ref, got):
        if a is not None:
            assert np.array_equal(to_host(a), to_host(b))


@pytest.mark.parametrize("n_tokens,H,E,k,T2", [
    (4096, 4096, 8, 2, 1000),        # the bench's batch shape, then a smaller batch
    (9000, 512, 256, 8, 77),         # many experts: the per-expert column scan
    (300, 64, 60, 4, 1),
])
def test_noalloc_matches_permute_on_two_calls(n_tokens, H, E, k, T2):
    g = np.random.default_rng(n_tokens + E)
    x = synth.bf16_bits(g.standard_normal((n_tokens, H)).astype(np.float32))
    idx = synth.random_topk_idx(n_tokens, E, k, seed=E + k)
    x_d, idx_d = to_dev(x), to_dev(idx)
    # first call: every token in a shuffled order; second: a smaller batch
    tok1 = g.permutation(n_tokens).astype(np.int32)
    tok2 = g.choice(n_tokens, size=T2, replace=False).astype(np.int32)
    _pair(x_d, idx_d, E, to_dev(tok1), n_tokens)
    _pair(x_d, idx_d, E, to_dev(tok2), T2)
    _pair(None, idx_d, E, None, n_tokens)           # maps only, all tokens in order

