"""Pins of the expert FFN oracle: matrix form against explicit loops, SiLU
special values, and the resident / missed split."""
import math

import numpy as np

import oracle
from paper_2410_17954_amd import synth


def test_silu_special_values():
    assert oracle.silu(0.0) == 0.0
    assert abs(oracle.silu(1.0) - 1.0 / (1.0 + math.exp(-1.0))) < 1e-16
    assert abs(oracle.silu(40.0) - 40.0) < 1e-12
    assert abs(oracle.silu(-40.0)) < 1e-15
    # silu(-u) = silu(u) - u
    u = np.linspace(-5, 5, 11)
    assert np.allclose(oracle.silu(-u), oracle.silu(u) - u, atol=1e-15)


def test_swiglu_matrix_form_matches_loops():
    g = np.random.default_rng(0)
    H, F, M = 6, 5, 4
    x = g.standard_normal((M, H))
    wg, wu, wd = g.standard_normal((F, H)), g.standard_normal((F, H)), g.standard_normal((H, F))
    assert np.allclose(oracle.swiglu(x, wg, wu, wd), oracle.swiglu_loops(x, wg, wu, wd),
                       rtol=1e-13, atol=1e-13)


def test_expert_ffn_tiny_config_against_loops():
    cfg = synth.workload("tiny_fp32")
    inp = synth.layer_inputs(cfg, seed=1, T=3, parts=("x", "experts"))
    x = inp["x"].astype(np.float64)
    e = 5
    ref = oracle.swiglu_loops(x, inp["w_gate"][e], inp["w_up"][e], inp["w_down"][e])
    offsets = np.array([0, 0, 0, 0, 0, 0, 3, 3, 3])
    slot = np.arange(8)
    y, computed = oracle.expert_ffn(x, offsets, slot, inp["w_gate"], inp["w_up"], inp["w_down"])
    assert computed.all()
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-14)


def test_non_resident_rows_are_not_computed():
    g = np.random.default_rng(1)
    E, H, F = 3, 4, 6
    wg, wu, wd = g.standard_normal((2, F, H)), g.standard_normal((2, F, H)), g.standard_normal((2, H, F))
    x = g.standard_normal((7, H))
    offsets = np.array([0, 2, 5, 7])
    slot = np.array([1, -1, 0])     # expert 0 -> slot 1, expert 1 missing, expert 2 -> slot 0
    y, computed = oracle.expert_ffn(x, offsets, slot, wg, wu, wd)
    assert computed.tolist() == [True, True, False, False, False, True, True]
    assert np.isnan(y[2:5]).all()
    assert np.allclose(y[0:2], oracle.swiglu(x[0:2], wg[1], wu[1], wd[1]))
    assert np.allclose(y[5:7], oracle.swiglu(x[5:7], wg[0], wu[0], wd[0]))
