"""Host <-> device plumbing shared by the GPU parity tests (no arithmetic of
the method lives here)."""
import numpy as np
import torch

from paper_2410_17954_amd import synth

DEV = "cuda:0"
U = 2.0 ** -24


def to_dev(a):
    """numpy -> device tensor; uint16 arrays are bf16 bit patterns."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(DEV)
    return torch.from_numpy(a).to(DEV)


def to_host(t):
    """device tensor -> numpy; bf16 comes back as uint16 bit patterns."""
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def vals(t):
    """Exact float64 values of a device tensor."""
    return synth.values(to_host(t))


def gamma(n):
    return n * U / (1 - n * U)


def rel_max_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    m = np.max(np.abs(ref))
    return float(np.max(np.abs(got - ref)) / (m if m > 0 else 1.0))


def logit_bound(x, w, z, bias=None):
    """Rigorous bound on |z_gpu - z_exact| for float32 accumulation of H
    exact bf16 products in any order (doubled for the fused accumulation of
    the matrix cores), plus the rounding of the bias add."""
    S = np.abs(x) @ np.abs(w).T
    H = x.shape[1]
    b = 0.0 if bias is None else np.abs(bias if np.ndim(bias) == 2 else bias[None, :])
    return 2 * gamma(H) * S + 2 * U * 2 * (np.abs(z) + b)


def check_topk_against_bound(idx_gpu, z, bound, k):
    """Indices must equal the exact top-k wherever the exact logits separate
    the first k+1 by more than twice the bound; elsewhere the GPU choice must
    be a valid top-k of some logits within the bound. Returns the number of
    near-tie tokens."""
    T, E = z.shape
    order = np.argsort(-z, axis=1, kind="stable")
    zs = np.take_along_axis(z, order, 1)
    bmax = bound.max(axis=1)
    kk = min(k + 1, E)
    gaps = -np.diff(zs[:, :kk], axis=1) if kk > 1 else np.full((T, 1), np.inf)
    sure = (gaps > 2 * bmax[:, None]).all(axis=1)
    assert np.array_equal(idx_gpu[sure], order[sure, :k]), "decided top-k differs"
    near = np.nonzero(~sure)[0]
    for t in near:
        sel = idx_gpu[t]
        assert len(set(sel.tolist())) == k and (sel >= 0).all() and (sel < E).all()
        tol = 2 * bmax[t]
        for j in range(k - 1):
            assert z[t, sel[j]] >= z[t, sel[j + 1]] - tol
        rest = np.setdiff1d(np.arange(E), sel)
        if rest.size:
            assert z[t, rest].max() <= z[t, sel[-1]] + tol
    return int(near.size)
