"""CPU checks of the C ABI: the library loads, exports every declared entry
point, and rejects invalid arguments on the host before touching a device."""
import ctypes
import os
import re

import pytest

from paper_2410_17954_amd import ops
from paper_2410_17954_amd.build import library_path

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moeflow.h")
FAKE = ctypes.c_void_p(0x1000)      # never dereferenced: validation fails first


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(library_path()):
        from paper_2410_17954_amd import build
        build.build(verbose=False)
    return ops.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(moe_\w+)\s*\(", text, re.M)))


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert len(names) == 33, names
    assert sorted(ops.exported_symbols()) == names
    for n in names:
        assert hasattr(lib, n)


def test_version_and_status_strings(lib):
    assert lib.moe_abi_version() == 2
    for s in range(5):
        assert lib.moe_status_str(s)
    assert lib.moe_status_str(99) == b"unknown status"


def test_workspace_queries(lib):
    assert lib.moe_permute_workspace(0, 2, 8) == 0
    assert lib.moe_permute_workspace(4096, 2, 8) % 256 == 0
    assert lib.moe_expert_ffn_workspace(8192, 4096, 14336, 8, 1) >= 8192 * 14336 * 2
    assert lib.moe_schedule_workspace(8192, 32, 8, 2) > 8192 * 4 * 8
    # the B-way workspace holds the largest split's plus a gathered copy of the routes
    assert (lib.moe_schedule_multi_workspace(8192, 32, 8, 2, 4)
            >= lib.moe_schedule_workspace(8192, 32, 8, 2) + 8192 * 32 * 2)
    assert lib.moe_schedule_multi_workspace(8192, 32, 8, 2, 0) == 0
    assert lib.moe_schedule_multi_workspace(8192, 32, 8, 2, 5000) == 0


def test_schedule_multi_rejects_bad_arguments(lib):
    S = None
    ws = lib.moe_schedule_multi_workspace(16, 2, 8, 2, 4)
    args = lambda N, E, k, B, perm=FAKE, off=FAKE, it=3, keep=1, nbytes=ws: lib.moe_schedule_multi(
        FAKE, N, 2, E, k, B, it, keep, perm, off, S, S, S, FAKE, nbytes, S)
    assert args(0, 8, 2, 4) == ops.MOE_ERR_ARG            # no tokens
    assert args(16, 8, 2, 0) == ops.MOE_ERR_ARG           # no batches
    assert args(16, 8, 2, 4097) == ops.MOE_ERR_ARG        # too many batches
    assert args(16, 8, 9, 4) == ops.MOE_ERR_ARG           # k > E
    assert args(16, 300, 2, 4) == ops.MOE_ERR_ARG         # E > 256
    assert args(16, 8, 2, 4, perm=S) == ops.MOE_ERR_ARG   # missing output
    assert args(16, 8, 2, 4, off=S) == ops.MOE_ERR_ARG
    assert args(16, 8, 2, 4, it=0) == ops.MOE_ERR_ARG
    assert args(16, 8, 2, 4, keep=2) == ops.MOE_ERR_ARG
    assert args(16, 8, 2, 4, nbytes=ws - 1) == ops.MOE_ERR_WORKSPACE


def test_route_rejects_bad_arguments(lib):
    S = None
    # T = 0, k > E, E > 256, missing outputs, bad bias mode, bf16 H % 8 != 0
    assert lib.moe_route(FAKE, FAKE, 1, 0, 64, 8, 2, S, 0, 1, S, FAKE, FAKE, S) == ops.MOE_ERR_ARG
    assert lib.moe_route(FAKE, FAKE, 1, 4, 64, 2, 3, S, 0, 1, S, FAKE, FAKE, S) == ops.MOE_ERR_ARG
    assert lib.moe_route(FAKE, FAKE, 1, 4, 64, 300, 3, S, 0, 1, S, FAKE, FAKE, S) == ops.MOE_ERR_ARG
    assert lib.moe_route(FAKE, FAKE, 1, 4, 64, 8, 2, S, 0, 1, S, S, FAKE, S) == ops.MOE_ERR_ARG
    assert lib.moe_route(FAKE, FAKE, 1, 4, 64, 8, 2, S, 1, 1, S, FAKE, FAKE, S) == ops.MOE_ERR_ARG
    assert lib.moe_route(FAKE, FAKE, 1, 4, 60, 8, 2, S, 0, 1, S, FAKE, FAKE, S) == ops.MOE_ERR_UNSUPPORTED
    assert lib.moe_route(FAKE, FAKE, 7, 4, 64, 8, 2, S, 0, 1, S, FAKE, FAKE, S) == ops.MOE_ERR_ARG
    # logits-in mode needs logits and no bias
    assert lib.moe_route(S, S, 1, 4, 0, 8, 2, S, 0, 1, S, FAKE, FAKE, S) == ops.MOE_ERR_ARG


def test_schedule_rejects_bad_arguments(lib):
    S = None
    ok = (FAKE, 64, 4, 8, 2, 32, 10, 1, FAKE, FAKE, FAKE, S)
    bad_n1 = (FAKE, 64, 4, 8, 2, 65, 10, 1, FAKE, FAKE, FAKE, S)
    assert lib.moe_schedule(*bad_n1, FAKE, 1 << 20, S) == ops.MOE_ERR_ARG
    assert lib.moe_schedule(FAKE, 64, 4, 8, 2, 32, 0, 1, FAKE, FAKE, FAKE, S, FAKE, 1 << 20, S) == ops.MOE_ERR_ARG
    assert lib.moe_schedule(FAKE, 64, 4, 8, 9, 32, 10, 1, FAKE, FAKE, FAKE, S, FAKE, 1 << 20, S) == ops.MOE_ERR_ARG
    assert lib.moe_schedule(S, 64, 4, 8, 2, 32, 10, 1, FAKE, FAKE, FAKE, S, FAKE, 1 << 20, S) == ops.MOE_ERR_ARG
    assert lib.moe_schedule(*ok, S, 0, S) == ops.MOE_ERR_WORKSPACE
    assert lib.moe_schedule(*ok, FAKE, 16, S) == ops.MOE_ERR_WORKSPACE
    assert lib.moe_schedule(*ok, ctypes.c_void_p(0x1001), 1 << 20, S) == ops.MOE_ERR_WORKSPACE


def test_permute_rejects_bad_arguments(lib):
    S = None
    assert lib.moe_permute(FAKE, 1, 64, 10, S, 10, FAKE, 2, 8, FAKE, FAKE, FAKE, S, FAKE, 1 << 20, S) == ops.MOE_ERR_ARG
    assert lib.moe_permute(FAKE, 1, 60, 10, S, 10, FAKE, 2, 8, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, S) == ops.MOE_ERR_UNSUPPORTED
    assert lib.moe_permute(FAKE, 1, 64, 5, S, 10, FAKE, 2, 8, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, S) == ops.MOE_ERR_ARG
    assert lib.moe_permute(FAKE, 1, 64, 10, S, 10, FAKE, 2, 8, FAKE, FAKE, FAKE, FAKE, FAKE, 8, S) == ops.MOE_ERR_WORKSPACE


def test_expert_ffn_rejects_bad_arguments(lib):
    S = None
    args = lambda dt, H, F, E, slot, nS, ws, wsb: (FAKE, dt, 128, H, F, FAKE, E, slot, nS, FAKE,
                                                  FAKE, FAKE, FAKE, ws, wsb, S)
    big = 1 << 30
    assert lib.moe_expert_ffn(*args(1, 60, 64, 4, FAKE, 4, FAKE, big)) == ops.MOE_ERR_UNSUPPORTED
    assert lib.moe_expert_ffn(*args(1, 64, 60, 4, FAKE, 4, FAKE, big)) == ops.MOE_ERR_UNSUPPORTED
    assert lib.moe_expert_ffn(*args(1, 64, 64, 4, S, 3, FAKE, big)) == ops.MOE_ERR_ARG
    assert lib.moe_expert_ffn(*args(1, 64, 64, 0, FAKE, 3, FAKE, big)) == ops.MOE_ERR_ARG
    assert lib.moe_expert_ffn(*args(5, 64, 64, 4, FAKE, 3, FAKE, big)) == ops.MOE_ERR_ARG
    assert lib.moe_expert_ffn(*args(1, 64, 64, 4, FAKE, 3, FAKE, 100)) == ops.MOE_ERR_WORKSPACE


def test_combine_rejects_bad_arguments(lib):
    S = None
    assert lib.moe_combine(FAKE, 1, 64, 10, S, 5, 5, 2, FAKE, FAKE, FAKE, S, 0, S, 2, FAKE, S, S) == ops.MOE_ERR_ARG
    assert lib.moe_combine(FAKE, 1, 60, 10, S, 5, 5, 2, FAKE, FAKE, FAKE, S, 0, S, 0, FAKE, S, S) == ops.MOE_ERR_UNSUPPORTED
    assert lib.moe_combine(FAKE, 1, 64, 10, S, 5, 5, 2, FAKE, FAKE, FAKE, FAKE, 0, S, 0, FAKE, S, S) == ops.MOE_ERR_ARG
    assert lib.moe_combine(S, 1, 64, 10, S, 5, 5, 2, FAKE, FAKE, FAKE, S, 0, S, 0, FAKE, S, S) == ops.MOE_ERR_ARG


def test_plan_slots_host_rule(lib):
    import numpy as np
    import oracle
    slot = ops.plan_slots(np.array([5, 0, 9, 5, 1]), 3)
    assert slot.tolist() == [0, -1, 1, 2, -1]
    assert ops.plan_slots(np.array([1, 2]), 0).tolist() == [-1, -1]
    assert ops.plan_slots(np.array([1, 2]), -3).tolist() == [-1, -1]
    assert ops.plan_slots(np.array([1, 2]), 5).tolist() == [0, 1]
    assert ops.plan_slots(np.zeros(6, np.int32), 2).tolist() == [0, 1, -1, -1, -1, -1]
    # the library's rule against the oracle's on random demand with many ties
    g = np.random.default_rng(3)
    for _ in range(200):
        E = int(g.integers(1, 70))
        d = g.integers(0, 5, size=E)
        S = int(g.integers(-1, E + 3))
        assert ops.plan_slots(d, S).tolist() == oracle.plan_slots(d, S).tolist()
    S = None
    assert lib.moe_plan_slots(S, 4, 2, FAKE) == ops.MOE_ERR_ARG
    assert lib.moe_plan_slots(FAKE, 0, 2, FAKE) == ops.MOE_ERR_ARG


def test_kv_and_stack_reject_bad_arguments(lib):
    S = None
    one = (ctypes.c_int64 * 1)(10)
    ptrs = (ctypes.c_void_p * 1)(0x1000)
    # no sources, 17 sources, merge with n_out != total, missing err
    assert lib.moe_kv_gather(ptrs, one, 0, 2, 64, S, 10, FAKE, FAKE, S) == ops.MOE_ERR_ARG
    assert lib.moe_kv_gather(ptrs, one, 17, 2, 64, S, 10, FAKE, FAKE, S) == ops.MOE_ERR_ARG
    assert lib.moe_kv_gather(ptrs, one, 1, 2, 64, S, 9, FAKE, FAKE, S) == ops.MOE_ERR_ARG
    assert lib.moe_kv_gather(ptrs, one, 1, 2, 64, S, 10, FAKE, S, S) == ops.MOE_ERR_ARG
    assert lib.moe_kv_reindex(FAKE, 0, FAKE, 2, FAKE, FAKE, FAKE, S) == ops.MOE_ERR_ARG
    assert lib.moe_kv_reindex(FAKE, 10, FAKE, 2, S, S, FAKE, S) == ops.MOE_ERR_ARG
    w = (ctypes.c_void_p * 2)(0x1000, 0x1000)
    ws = lib.moe_stack_workspace(16, 64, 64, 8, 2, 1)
    call = (lambda T=16, n=16, E=8, k=2, S_=8, slot=S, tok=S, nbytes=ws, wr=w, pre=0, nw=S,
            eps=1e-5: lib.moe_stack_forward(FAKE, 1, n, 64, tok, T, 2, E, k, 64, wr, w, w, w, slot,
                                            S_, 1, pre, nw, eps, S, S, FAKE, FAKE, nbytes, S))
    assert call(T=0) == ops.MOE_ERR_ARG
    assert call(n=20) == ops.MOE_ERR_ARG                  # n_tokens != T without token ids
    assert call(k=9) == ops.MOE_ERR_ARG
    assert call(S_=4) == ops.MOE_ERR_ARG                  # S < E needs a slot table
    assert call(wr=(ctypes.c_void_p * 2)(0x1000, 0)) == ops.MOE_ERR_ARG
    assert call(nbytes=ws - 1) == ops.MOE_ERR_WORKSPACE
    assert call(pre=0, nw=w) == ops.MOE_ERR_ARG            # norm weights without the norm
    assert call(pre=1, eps=-1.0) == ops.MOE_ERR_ARG
    assert call(pre=2) == ops.MOE_ERR_ARG
    assert call(pre=1, nw=(ctypes.c_void_p * 2)(0x1000, 0)) == ops.MOE_ERR_ARG


def test_rpp_weight_count_and_bad_arguments(lib):
    dims = dict(vocab=32000, d_model=32, n_heads=4, d_ff=2048, n_enc=3, n_dec=3, L=32, E=8,
                num_buckets=32, max_distance=128, eps=1e-6)
    g = ops.rpp_dims(dims)
    # the library's own count of the packed layout (7.43 MB in float32)
    assert lib.moe_rpp_weights_count(ctypes.byref(g)) == 1856288
    assert lib.moe_rpp_workspace(16, 512, ctypes.byref(g)) > 16 * 512 * 2048 * 4
    S = None
    ws = lib.moe_rpp_workspace(2, 8, ctypes.byref(g))
    call = lambda B=2, S_=8, gg=g, nbytes=ws: lib.moe_rpp_forward(
        FAKE, B, S_, ctypes.byref(gg), FAKE, FAKE, S, FAKE, FAKE, nbytes, S)
    assert call(B=0) == ops.MOE_ERR_ARG
    assert call(S_=0) == ops.MOE_ERR_ARG
    bad = ops.rpp_dims(dict(dims, n_heads=5))           # d_model % n_heads != 0
    assert lib.moe_rpp_weights_count(ctypes.byref(bad)) == 0
    assert call(gg=bad) == ops.MOE_ERR_ARG
    odd = ops.rpp_dims(dict(dims, max_distance=100))    # not a power of two
    assert call(gg=odd, nbytes=lib.moe_rpp_workspace(2, 8, ctypes.byref(odd))) == \
        ops.MOE_ERR_UNSUPPORTED
    assert call(nbytes=ws - 1) == ops.MOE_ERR_WORKSPACE


def test_permute_noalloc_rejects_on_the_host(lib):
    S = None
    # beyond the static scratch (300000 tokens, 256 experts, top-8)
    assert lib.moe_permute_workspace(300000, 8, 256) > 4 * 1024 * 1024
    assert lib.moe_permute_noalloc(S, 0, 0, 300000, S, 300000, FAKE, 8, 256, FAKE, FAKE, FAKE, S,
                                   S) == ops.MOE_ERR_WORKSPACE
    # the argument rules of moe_permute
    assert lib.moe_permute_noalloc(S, 0, 0, 10, S, 10, S, 2, 8, FAKE, FAKE, FAKE, S, S) == ops.MOE_ERR_ARG
    assert lib.moe_permute_noalloc(S, 0, 0, 10, S, 10, FAKE, 9, 8, FAKE, FAKE, FAKE, S, S) == ops.MOE_ERR_ARG
    assert lib.moe_permute_noalloc(FAKE, 1, 64, 10, S, 10, FAKE, 2, 8, FAKE, FAKE, FAKE, S, S) == ops.MOE_ERR_ARG
    assert lib.moe_permute_noalloc(FAKE, 1, 60, 10, S, 10, FAKE, 2, 8, FAKE, FAKE, FAKE, FAKE, S) == ops.MOE_ERR_UNSUPPORTED


def test_route_binarize_rejects_on_the_host(lib):
    S = None
    assert lib.moe_route_binarize(S, 10, 8, 2, FAKE, S) == ops.MOE_ERR_ARG
    assert lib.moe_route_binarize(FAKE, 10, 8, 2, S, S) == ops.MOE_ERR_ARG
    assert lib.moe_route_binarize(FAKE, 0, 8, 2, FAKE, S) == ops.MOE_ERR_ARG
    assert lib.moe_route_binarize(FAKE, 10, 8, 9, FAKE, S) == ops.MOE_ERR_ARG
    assert lib.moe_route_binarize(FAKE, 10, 257, 2, FAKE, S) == ops.MOE_ERR_ARG


def test_probe_copy_rejects_on_the_host(lib):
    # validated before any launch: null buffers, a size that is not a
    # multiple of 16, a misaligned buffer (the pointers are never touched)
    fake = ctypes.c_void_p(4096)
    assert lib.moe_probe_copy(None, fake, 16, None) != 0
    assert lib.moe_probe_copy(fake, fake, 24, None) != 0
    assert lib.moe_probe_copy(ctypes.c_void_p(4104), fake, 16, None) != 0
    assert lib.moe_probe_copy(fake, fake, 0, None) != 0


def test_one_hip_runtime_whatever_the_import_order(lib):
    """Loading the library before torch must not bring a second HIP runtime
    into the process (torch names the runtime without its version, the
    library with it): the binding loads torch's first."""
    import subprocess
    import sys
    code = ("import sys; sys.path.insert(0, %r)\n"
            "from paper_2410_17954_amd import ops\n"
            "ops.load_library()\n"
            "import torch\n"
            "maps = open('/proc/self/maps').read().splitlines()\n"
            "print(len({l.split()[-1] for l in maps if 'libamdhip64' in l}))\n") % ROOT
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                         timeout=300)
    assert out.returncode == 0, out.stderr[-2000:]
    assert out.stdout.strip().splitlines()[-1] == "1"
