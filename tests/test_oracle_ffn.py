"""Pins for the oracle's expert arithmetic (CPU only): closed forms of silu
and of the SwiGLU expert, and the structure of Eq. (1)."""

import json
import math
import os

import numpy as np
import pytest

from conftest import GOLDEN
from oracle import combine, moe_output, silu, swiglu_ffn


def test_silu_closed_forms():
    assert silu(0.0) == 0.0
    assert silu(1.0) == pytest.approx(1.0 / (1.0 + math.exp(-1.0)), rel=1e-15)
    assert silu(-2.0) == pytest.approx(-2.0 / (1.0 + math.exp(2.0)), rel=1e-15)
    # silu -> identity for large z, -> 0 for very negative z
    assert silu(50.0) == pytest.approx(50.0, rel=1e-15)
    assert abs(silu(-800.0)) == 0.0
    # silu(z) - silu(-z) = z
    z = np.linspace(-5, 5, 11)
    assert np.allclose(silu(z) - silu(-z), z, rtol=0, atol=1e-14)


def test_swiglu_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "swiglu_closed_form.json")))
    out = swiglu_ffn(np.array([g["v"]]), np.array(g["w_gate"], float),
                     np.array(g["w_up"], float), np.array(g["w_down"], float))
    assert out.shape == (1, 2)
    assert np.allclose(out[0], g["expected"], rtol=1e-15, atol=0)


def test_swiglu_scalar_and_roles():
    # D = F = 1: FFN(x) = silu(a x) * (b x) * c
    a, b, c, x = 0.7, -1.3, 2.5, 0.9
    want = (a * x) / (1 + math.exp(-a * x)) * (b * x) * c
    got = swiglu_ffn(np.array([[x]]), np.array([[a]]), np.array([[b]]),
                     np.array([[c]]))[0, 0]
    assert got == pytest.approx(want, rel=1e-15)
    # gate and up play different roles: swapping them changes the value
    swapped = swiglu_ffn(np.array([[x]]), np.array([[b]]), np.array([[a]]),
                         np.array([[c]]))[0, 0]
    assert abs(swapped - want) > 1e-3


def test_swiglu_is_rowwise():
    rng = np.random.default_rng(3)
    D, F = 5, 7
    wg, wu, wd = rng.normal(size=(D, F)), rng.normal(size=(D, F)), rng.normal(size=(F, D))
    v = rng.normal(size=(4, D))
    full = swiglu_ffn(v, wg, wu, wd)
    for i in range(4):
        assert np.allclose(full[i], swiglu_ffn(v[i:i + 1], wg, wu, wd)[0],
                           rtol=1e-13, atol=1e-13)
    # the zero vector maps to zero; a zero down-projection gives zero
    assert np.all(swiglu_ffn(np.zeros((1, D)), wg, wu, wd) == 0)
    assert np.all(swiglu_ffn(v, wg, wu, np.zeros((F, D))) == 0)


def _expert_bank():
    """Expert 0 is the worked example; expert 1 maps v to zero; expert 2 is
    the worked example scaled by 2 in the down projection."""
    g = json.load(open(os.path.join(GOLDEN, "swiglu_closed_form.json")))
    wg, wu, wd = (np.array(g[k], float) for k in ("w_gate", "w_up", "w_down"))
    bank = {0: (wg, wu, wd), 1: (wg, wu, 0 * wd), 2: (wg, wu, 2 * wd)}
    return bank, np.array(g["expected"])


def test_moe_output_gate_weighted_sum():
    bank, f0 = _expert_bank()
    x = np.array([[1.0, 2.0], [1.0, 2.0], [1.0, 2.0]])
    ids = np.array([[0, 1], [1, 2], [2, 2]])
    gates = np.array([[0.25, 0.75], [0.6, 0.4], [0.3, 0.7]], dtype=np.float32)
    y = moe_output(x, ids, gates, lambda e: bank[e])
    assert np.allclose(y[0], 0.25 * f0, rtol=1e-15)
    assert np.allclose(y[1], np.float64(np.float32(0.4)) * 2 * f0, rtol=1e-15)
    # an expert repeated inside a token counts once per pair
    assert np.allclose(y[2], (np.float64(np.float32(0.3)) + np.float64(np.float32(0.7))) * 2 * f0,
                       rtol=1e-14)


def test_moe_output_token_subset_and_bad_ids():
    rng = np.random.default_rng(0)
    E, D, F, T, K = 4, 6, 5, 9, 2
    W = {e: (rng.normal(size=(D, F)), rng.normal(size=(D, F)), rng.normal(size=(F, D)))
         for e in range(E)}
    x = rng.normal(size=(T, D))
    ids = rng.integers(0, E, size=(T, K))
    gates = rng.random((T, K)).astype(np.float32)
    full = moe_output(x, ids, gates, lambda e: W.get(e))
    sub = moe_output(x, ids, gates, lambda e: W.get(e), tokens=[7, 2])
    assert np.allclose(sub, full[[7, 2]], rtol=1e-13, atol=1e-13)
    # gates scale linearly
    assert np.allclose(moe_output(x, ids, 2 * gates, lambda e: W.get(e)), 2 * full,
                       rtol=1e-14, atol=0)
    # a pair with an out-of-range id contributes nothing
    ids2 = ids.copy()
    ids2[0, 1] = E + 3
    y2 = moe_output(x, ids2, gates, lambda e: W.get(e))
    want = np.float64(gates[0, 0]) * swiglu_ffn(x[:1], *W[ids[0, 0]])[0]
    assert np.allclose(y2[0], want, rtol=1e-14)


def test_combine_matches_moe_output_and_closed_form():
    bank, f0 = _expert_bank()
    x = np.array([[1.0, 2.0], [1.0, 2.0]])
    ids = np.array([[0, 2], [1, 0]])
    gates = np.array([[0.5, 0.25], [1.0, 2.0]], dtype=np.float32)
    pair_out = np.stack([np.stack([swiglu_ffn(x[t:t + 1], *bank[ids[t, k]])[0] for k in range(2)])
                         for t in range(2)])
    y = combine(pair_out, gates)
    assert np.allclose(y[0], 0.5 * f0 + 0.25 * 2 * f0, rtol=1e-15)
    assert np.allclose(y[1], 2.0 * f0, rtol=1e-15)
    assert np.allclose(y, moe_output(x, ids, gates, lambda e: bank[e]), rtol=1e-14)
