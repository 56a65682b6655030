"""Pins of the backward oracle: central finite differences of the forward
definitions (float64), scalar closed forms, and the plan-based gradients
(with the gradient return) equal to the plan-free ones under LLEP and EP."""

import math

import numpy as np
import pytest

import oracle
from oracle.backward import (combine_backward, moe_backward, plan_backward, silu_grad,
                             swiglu_ffn_backward)

EPS = 1e-6


def _num_grad(f, a):
    """Central differences of the scalar f() with respect to every entry of a."""
    g = np.zeros_like(a)
    it = np.nditer(a, flags=["multi_index"])
    for _ in it:
        i = it.multi_index
        old = a[i]
        a[i] = old + EPS
        hi = f()
        a[i] = old - EPS
        lo = f()
        a[i] = old
        g[i] = (hi - lo) / (2 * EPS)
    return g


def test_silu_grad_finite_differences():
    z = np.linspace(-8, 8, 33)
    num = (oracle.silu(z + EPS) - oracle.silu(z - EPS)) / (2 * EPS)
    assert np.allclose(silu_grad(z), num, rtol=1e-7, atol=1e-9)
    # closed forms: silu'(0) = 1/2, silu' -> 1 for large z, -> 0 for very negative z
    assert silu_grad(0.0) == pytest.approx(0.5)
    assert silu_grad(40.0) == pytest.approx(1.0)
    assert abs(silu_grad(-40.0)) < 1e-15


@pytest.mark.parametrize("seed", [0, 1])
def test_swiglu_backward_finite_differences(seed):
    rng = np.random.default_rng(seed)
    n, D, F = 3, 4, 5
    v, wg, wu = rng.normal(size=(n, D)), rng.normal(size=(D, F)), rng.normal(size=(D, F))
    wd, d_out = rng.normal(size=(F, D)), rng.normal(size=(n, D))

    def loss():
        return float(np.sum(d_out * oracle.swiglu_ffn(v, wg, wu, wd)))

    dv, dwg, dwu, dwd = swiglu_ffn_backward(v, wg, wu, wd, d_out)
    for got, a in ((dv, v), (dwg, wg), (dwu, wu), (dwd, wd)):
        assert np.allclose(got, _num_grad(loss, a), rtol=1e-6, atol=1e-7)


def test_swiglu_backward_scalar_closed_form():
    # D = F = 1: out = silu(v a) (v b) c
    v, a, b, c, dout = 0.7, -1.3, 0.4, 2.1, 1.5
    s = 1 / (1 + math.exp(-v * a))
    silu = v * a * s
    dsilu = s * (1 + v * a * (1 - s))
    want_dv = dout * c * (dsilu * a * (v * b) + silu * b)
    want_da = dout * c * dsilu * v * (v * b)
    want_db = dout * c * silu * v
    want_dc = dout * silu * (v * b)
    dv, dwg, dwu, dwd = swiglu_ffn_backward(np.array([[v]]), np.array([[a]]), np.array([[b]]),
                                            np.array([[c]]), np.array([[dout]]))
    assert dv[0, 0] == pytest.approx(want_dv, rel=1e-12)
    assert dwg[0, 0] == pytest.approx(want_da, rel=1e-12)
    assert dwu[0, 0] == pytest.approx(want_db, rel=1e-12)
    assert dwd[0, 0] == pytest.approx(want_dc, rel=1e-12)


def test_combine_backward_finite_differences():
    rng = np.random.default_rng(4)
    T, K, D = 3, 2, 4
    pair_out, gates, dy = rng.normal(size=(T, K, D)), rng.normal(size=(T, K)), rng.normal(size=(T, D))

    def loss():
        return float(np.sum(dy * oracle.combine(pair_out, gates)))

    dpo, dg = combine_backward(dy, pair_out, gates)
    assert np.allclose(dpo, _num_grad(loss, pair_out), rtol=1e-6, atol=1e-8)
    assert np.allclose(dg, _num_grad(loss, gates), rtol=1e-6, atol=1e-8)


def _tiny_layer(seed, T=6, K=2, E=4, D=3, F=4, bad=False):
    rng = np.random.default_rng(seed)
    ids = rng.integers(0, E, (T, K))
    if bad:
        ids[1, 0] = E  # an invalid id: contributes nothing
    gates = rng.normal(size=(T, K))
    x = rng.normal(size=(T, D))
    W = {e: (rng.normal(size=(D, F)), rng.normal(size=(D, F)), rng.normal(size=(F, D)))
         for e in range(E)}
    dy = rng.normal(size=(T, D))
    return ids, gates, x, W, dy


@pytest.mark.parametrize("bad", [False, True])
def test_moe_backward_finite_differences(bad):
    ids, gates, x, W, dy = _tiny_layer(7, bad=bad)
    E = 4

    def loss():
        return float(np.sum(dy * oracle.moe_output(x, ids, gates, lambda e: W.get(e))))

    dx, dgates, dW = moe_backward(x, ids, gates, lambda e: W[e], dy, E)
    assert np.allclose(dx, _num_grad(loss, x), rtol=1e-6, atol=1e-7)
    assert np.allclose(dgates, _num_grad(loss, gates), rtol=1e-6, atol=1e-7)
    for e, (dwg, dwu, dwd) in dW.items():
        for got, a in ((dwg, W[e][0]), (dwu, W[e][1]), (dwd, W[e][2])):
            assert np.allclose(got, _num_grad(loss, a), rtol=1e-6, atol=1e-7)
    if bad:
        assert dgates[1, 0] == 0.0


@pytest.mark.parametrize("mode,cap,m", [("llep", 3, 1), ("llep", 2, 2), ("llep", 4, 1),
                                        ("ep", 3, 1)])
def test_plan_backward_equals_plan_free(mode, cap, m):
    """Through any plan (spills, force-assigns, or EP), the gradients with the
    gradient return equal the plan-free ones; EP keeps every partial native."""
    T, K, E, P = 9, 2, 4, 2
    ids, gates, x, W, dy = _tiny_layer(11, T=T, K=K, E=E)
    ids[:, 0] = 0  # expert 0 overloaded: its load spills under LLEP
    flat = ids.reshape(-1).tolist()
    pl = oracle.plan(flat, E, P, cap, m, mode=mode)
    _, row_pair = oracle.permute(flat, pl, E)
    dx_p, partials, dW_p = plan_backward(x, np.array(flat), gates.reshape(-1), lambda e: W[e],
                                         dy, pl, np.asarray(row_pair), K, E // P)
    dx, _, dW = moe_backward(x, ids, gates, lambda e: W[e], dy, E)
    assert np.allclose(dx_p, dx, rtol=1e-12, atol=1e-12)
    assert sorted(dW_p) == sorted(dW)
    for e in dW:
        for a, b in zip(dW_p[e], dW[e]):
            assert np.allclose(a, b, rtol=1e-12, atol=1e-12)
    foreign = [(d, e) for (d, e) in partials if d != e // (E // P)]
    if mode == "ep":
        assert not foreign
    elif cap < math.ceil(T * K / P) + 2:
        assert foreign  # expert 0 spilled: some partials are returned
