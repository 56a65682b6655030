"""CPU oracle for the backward pass of the LLEP expert layer.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper states that LLEP is exact and supports gradient propagation: in the
backward pass the weight gradients computed for spilled chunks on foreign
devices are sent back to the expert's native device and added to the native
gradient (Sec. 4, "Elaboration"; Sec. 1). The functions below are the plain
definitions, in float64:

* `swiglu_ffn_backward`: gradients of FFN(v) = (silu(v Wg) * (v Wu)) Wd
  (Sec. 5.1, three matrices) for a block of rows, given d out;
* `combine_backward`: gradients of Eq. (1), y[t] = sum_k gate[t, k] out[t, k];
* `moe_backward`: the whole layer, plan-free (dx, d gates, per-expert dW);
* `plan_backward`: the same through a plan's groups: per group the rows'
  input and weight gradients, then the gradient return: each expert's
  weight gradient is the native device's partial plus the partials of the
  devices its load spilled to, added in increasing device order.

Pins: finite differences of the forward definitions, the EP and LLEP plans
giving the same gradients, and scalar closed forms (tests/test_oracle_backward.py).
"""

from __future__ import annotations

from typing import Dict, List, Optional, Tuple

import numpy as np

from .llep import PlanResult, silu


def silu_grad(z):
    """d/dz z * sigmoid(z) = sigmoid(z) * (1 + z * (1 - sigmoid(z)))."""
    z = np.asarray(z, dtype=np.float64)
    s = 1.0 / (1.0 + np.exp(-z))
    return s * (1.0 + z * (1.0 - s))


def swiglu_ffn_backward(v: np.ndarray, wg: np.ndarray, wu: np.ndarray, wd: np.ndarray,
                        d_out: np.ndarray):
    """Gradients of out = (silu(v Wg) * (v Wu)) Wd for rows v (n x D).

    Returns (dv [n x D], dWg [D x F], dWu [D x F], dWd [F x D]), float64:
      g = v Wg, u = v Wu, a = silu(g) * u
      da = d_out Wd^T
      dg = da * u * silu'(g),  du = da * silu(g)
      dv = dg Wg^T + du Wu^T
      dWg = v^T dg, dWu = v^T du, dWd = a^T d_out
    """
    v = np.asarray(v, dtype=np.float64)
    wg = np.asarray(wg, dtype=np.float64)
    wu = np.asarray(wu, dtype=np.float64)
    wd = np.asarray(wd, dtype=np.float64)
    d_out = np.asarray(d_out, dtype=np.float64)
    g = v @ wg
    u = v @ wu
    a = silu(g) * u
    da = d_out @ wd.T
    dg = da * u * silu_grad(g)
    du = da * silu(g)
    dv = dg @ wg.T + du @ wu.T
    return dv, v.T @ dg, v.T @ du, a.T @ d_out


def combine_backward(dy: np.ndarray, pair_out: np.ndarray, gates: np.ndarray):
    """Gradients of Eq. (1), y[t] = sum_k gates[t, k] * pair_out[t, k]:
    d pair_out[t, k] = gates[t, k] * dy[t]; d gates[t, k] = <dy[t], pair_out[t, k]>.
    dy: T x D; pair_out: T x K x D; gates: T x K."""
    dy = np.asarray(dy, dtype=np.float64)
    pair_out = np.asarray(pair_out, dtype=np.float64)
    gates = np.asarray(gates, dtype=np.float64)
    return gates[:, :, None] * dy[:, None, :], np.einsum("td,tkd->tk", dy, pair_out)


def moe_backward(x: np.ndarray, ids: np.ndarray, gates: np.ndarray, expert_weights,
                 dy: np.ndarray, E: int):
    """Plan-free gradients of the layer y = Eq. (1) with SwiGLU experts.

    Returns (dx [T x D], d_gates [T x K], dW: dict e -> (dWg, dWu, dWd)).
    Pairs with an id outside [0, E) contribute nothing (and get d gate 0).
    """
    x = np.asarray(x, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    T, K = ids.shape
    dx = np.zeros_like(x)
    dgates = np.zeros((T, K), dtype=np.float64)
    dW: Dict[int, Tuple[np.ndarray, np.ndarray, np.ndarray]] = {}
    by_expert: Dict[int, List[Tuple[int, int]]] = {}
    for t in range(T):
        for k in range(K):
            e = int(ids[t, k])
            if 0 <= e < E:
                by_expert.setdefault(e, []).append((t, k))
    for e, items in sorted(by_expert.items()):
        wg, wu, wd = expert_weights(e)
        toks = np.array([t for (t, _) in items])
        g = np.array([gates[t, k] for (t, k) in items], dtype=np.float64)
        v = x[toks]
        out = (silu(v @ np.asarray(wg, np.float64)) * (v @ np.asarray(wu, np.float64))) @ \
            np.asarray(wd, np.float64)
        d_out = g[:, None] * dy[toks]
        dv, dwg, dwu, dwd = swiglu_ffn_backward(v, wg, wu, wd, d_out)
        for j, (t, k) in enumerate(items):
            dx[t] += dv[j]
            dgates[t, k] = float(dy[t] @ out[j])
        dW[e] = (dwg, dwu, dwd)
    return dx, dgates, dW


def plan_backward(x: np.ndarray, ids_flat, gates_flat, expert_weights, dy: np.ndarray,
                  pl: PlanResult, row_pair: np.ndarray, K: int, M: int):
    """Gradients through the plan's groups, with the gradient return.

    For each group (device d, expert e, rows [s, s+n)) the rows' pairs are
    row_pair[s:s+n]; the group computes its rows' input gradients and a
    partial weight gradient of e from its rows only. Each expert's weight
    gradient is then the partial of its native device (d = e // M) plus the
    partials of the other devices in increasing device order.

    Returns (dx [T x D], partials: dict (d, e) -> (dWg, dWu, dWd),
    dW: dict e -> (dWg, dWu, dWd)).
    """
    x = np.asarray(x, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    dx = np.zeros_like(x)
    partials: Dict[Tuple[int, int], Tuple[np.ndarray, np.ndarray, np.ndarray]] = {}
    for (d, e, s, n) in pl.groups:
        pairs = row_pair[s:s + n]
        toks = pairs // K
        g = np.asarray(gates_flat, dtype=np.float64)[pairs]
        wg, wu, wd = expert_weights(e)
        dv, dwg, dwu, dwd = swiglu_ffn_backward(x[toks], wg, wu, wd, g[:, None] * dy[toks])
        np.add.at(dx, toks, dv)
        partials[(d, e)] = (dwg, dwu, dwd)
    dW: Dict[int, Tuple[np.ndarray, np.ndarray, np.ndarray]] = {}
    for e in sorted({e for (_, e) in partials}):
        native = e // M
        order = [native] + sorted(d for (d, ee) in partials if ee == e and d != native)
        acc = None
        for d in order:
            if (d, e) not in partials:
                continue
            p = partials[(d, e)]
            acc = tuple(q.copy() for q in p) if acc is None else tuple(a + q for a, q in zip(acc, p))
        dW[e] = acc
    return dx, partials, dW
