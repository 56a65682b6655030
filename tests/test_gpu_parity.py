"""GPU parity of the library against the oracle on small and ragged inputs:
the plan and the permutation bit-exactly, expert outputs within tolerance,
and the edge cases of the method."""

import json
import math
import os

import numpy as np
import pytest

import oracle
from conftest import GOLDEN
from gpu_util import LayerRun, assert_plan_equal, device, rel_err, report, run_plan

pytestmark = pytest.mark.gpu

TOL_BF16 = 2e-2
TOL_F32 = 1e-5


@pytest.fixture(scope="module")
def dev():
    return device()


def _ids_from_loads(loads, seed=0):
    rng = np.random.default_rng(seed)
    ids = np.concatenate([np.full(l, e, np.int32) for e, l in enumerate(loads)])
    return rng.permutation(ids).astype(np.int32)


# ---------------------------------------------------------------------------
# plan
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("trace", json.load(open(os.path.join(GOLDEN, "lla_hand_traces.json")))["traces"],
                         ids=lambda t: t["name"].split()[0])
def test_plan_hand_traces(dev, trace):
    loads, P = trace["loads"], trace["P"]
    E = len(loads)
    ids = _ids_from_loads(loads)
    got, info, _ = run_plan(ids[:, None], E, P, trace["cap"], trace["m"], dev=dev)
    ref = oracle.plan(ids.tolist(), E, P, trace["cap"], trace["m"])
    assert_plan_equal(got, info, ref)
    assert got["device_rows"] == trace["device_rows"]
    assert [list(t) for t in got["transfers"]] == trace["transfers"]


def _random_cases():
    rng = np.random.default_rng(1234)
    cases = []
    for i in range(40):
        P = int(rng.choice([1, 2, 3, 4, 8, 16]))
        M = int(rng.integers(1, 9))
        E = P * M
        K = int(rng.integers(1, 5))
        T = int(rng.integers(0, 3000))
        kind = i % 4
        if kind == 0:    # one hot expert
            ids = np.where(rng.random((T, K)) < 0.8, 0, rng.integers(0, E, (T, K)))
        elif kind == 1:  # zipf-like
            w = (np.arange(E) + 1.0) ** -1.3
            ids = rng.choice(E, size=(T, K), p=w / w.sum())
        elif kind == 2:  # uniform
            ids = rng.integers(0, E, (T, K))
        else:            # a few hot experts, some experts empty
            ids = rng.integers(0, max(1, E // 3), (T, K))
        R = T * K
        slack = [0, 0, 1, 7, R // 5][i % 5]
        cap = max(1, math.ceil(R / P) + slack)
        m = [1, 1, 3, 64][i % 4]
        cases.append((ids.astype(np.int32), E, P, cap, m))
    return cases


@pytest.mark.parametrize("case", _random_cases(), ids=lambda c: f"E{c[1]}P{c[2]}T{c[0].shape[0]}m{c[4]}")
def test_plan_random_matches_oracle(dev, case):
    ids, E, P, cap, m = case
    got, info, _ = run_plan(ids, E, P, cap, m, dev=dev)
    ref = oracle.plan(ids.reshape(-1).tolist(), E, P, cap, m)
    assert_plan_equal(got, info, ref)


def _tight_cases():
    """Many experts (several 64-expert blocks of the greedy loop), capacities
    below and above the balanced load, several spilling experts per block,
    experts whose native device is already over capacity (Case 3), and
    force-assigns (m > 1 or P * cap < R)."""
    rng = np.random.default_rng(777)
    cases = []
    shapes = [(96, 2), (96, 8), (192, 8), (192, 32), (320, 4), (320, 64), (512, 16), (512, 64)]
    for i in range(24):
        E, P = shapes[i % len(shapes)]
        T, K = int(rng.integers(500, 4000)), int(rng.choice([1, 4, 8]))
        kind = i % 3
        if kind == 0:    # zipf over a shuffled expert order
            w = (np.arange(E) + 1.0) ** -float(rng.uniform(0.8, 1.6))
            ids = rng.choice(E, size=(T, K), p=rng.permutation(w / w.sum()))
        elif kind == 1:  # a hot block of experts on a few devices
            hot = rng.choice(E, size=max(1, E // 16), replace=False)
            ids = np.where(rng.random((T, K)) < 0.7, rng.choice(hot, size=(T, K)),
                           rng.integers(0, E, (T, K)))
        else:            # experts of device 0 all heavy: Case 3 for some of them
            M = E // P
            ids = np.where(rng.random((T, K)) < 0.6, rng.integers(0, M, (T, K)),
                           rng.integers(0, E, (T, K)))
        R = T * K
        cap = max(1, int(math.ceil(R / P) * [0.5, 0.9, 1.0, 1.3][i % 4]))
        m = [1, 5, 50][i % 3]
        cases.append((ids.astype(np.int32), E, P, cap, m))
    return cases


@pytest.mark.parametrize("case", _tight_cases(),
                         ids=lambda c: f"E{c[1]}P{c[2]}R{c[0].size}cap{c[3]}m{c[4]}")
def test_plan_tight_capacity_matches_oracle(dev, case):
    ids, E, P, cap, m = case
    got, info, _ = run_plan(ids, E, P, cap, m, dev=dev)
    ref = oracle.plan(ids.reshape(-1).tolist(), E, P, cap, m)
    assert_plan_equal(got, info, ref)


def _repeated_chunk_cases():
    """Plans in which one expert has two or more chunks on the same device
    (an over-tight capacity sends force-assigned remainders back to devices
    that already hold a chunk of the expert): the table layout then has to
    merge chunks into one group and order them by start within it."""
    rng = np.random.default_rng(4242)
    cases = []
    while len(cases) < 12:
        P = int(rng.choice([2, 3, 4, 8]))
        M = int(rng.integers(1, 5))
        E = P * M
        T, K = int(rng.integers(200, 2500)), int(rng.integers(1, 4))
        hot = rng.choice(E, size=max(1, E // 4), replace=False)
        ids = np.where(rng.random((T, K)) < 0.7, rng.choice(hot, size=(T, K)),
                       rng.integers(0, E, (T, K))).astype(np.int32)
        cap = max(1, int(math.ceil(T * K / P) * float(rng.choice([0.3, 0.5]))))
        m = int(rng.choice([3, 50]))
        ref = oracle.plan(ids.reshape(-1).tolist(), E, P, cap, m)
        if len(ref.chunks) > len(ref.groups):
            cases.append((ids, E, P, cap, m))
    return cases


@pytest.mark.parametrize("case", _repeated_chunk_cases(),
                         ids=lambda c: f"E{c[1]}P{c[2]}R{c[0].size}cap{c[3]}m{c[4]}")
def test_plan_repeated_device_chunks_matches_oracle(dev, case):
    ids, E, P, cap, m = case
    got, info, _ = run_plan(ids, E, P, cap, m, dev=dev)
    ref = oracle.plan(ids.reshape(-1).tolist(), E, P, cap, m)
    assert len(ref.chunks) > len(ref.groups)
    assert_plan_equal(got, info, ref)


@pytest.mark.parametrize("E,P", [(512, 64), (512, 8), (256, 64)])
def test_plan_max_sizes(dev, E, P):
    rng = np.random.default_rng(E + P)
    T, K = 20000, 8
    w = (np.arange(E) + 1.0) ** -1.1
    ids = rng.choice(E, size=(T, K), p=w / w.sum()).astype(np.int32)
    cap = math.ceil(T * K / P)
    for mode in ("llep", "ep"):
        got, info, _ = run_plan(ids, E, P, cap, 1, mode=mode, dev=dev)
        ref = oracle.plan(ids.reshape(-1).tolist(), E, P, cap, 1, mode=mode)
        assert_plan_equal(got, info, ref)


def test_plan_lambda_bypass(dev):
    rng = np.random.default_rng(5)
    E, P, T, K = 32, 8, 4096, 4
    balanced = rng.permutation(np.repeat(np.arange(E), T * K // E)).reshape(T, K).astype(np.int32)
    skewed = np.where(rng.random((T, K)) < 0.5, 3, rng.integers(0, E, (T, K))).astype(np.int32)
    cap = math.ceil(T * K / P)
    for ids, lam in ((balanced, 1.3), (skewed, 1.3), (skewed, 1e9), (balanced, 1.0)):
        got, info, _ = run_plan(ids, E, P, cap, 1, lam=lam, dev=dev)
        ref = oracle.plan(ids.reshape(-1).tolist(), E, P, cap, 1, lam=lam)
        assert_plan_equal(got, info, ref)
    # balanced routing: LLEP yields the standard EP plan even without bypass
    got, info, _ = run_plan(balanced, E, P, cap, 1, dev=dev)
    ep, _, _ = run_plan(balanced, E, P, cap, 1, mode="ep", dev=dev)
    assert got["chunks"] == ep["chunks"] and got["groups"] == ep["groups"]


def test_plan_bad_ids_and_empty(dev):
    ids = np.array([[0, 1], [9, 2], [-1, 3], [7, 7]], np.int32)
    got, info, _ = run_plan(ids, 8, 2, 3, dev=dev)
    ref = oracle.plan(ids.reshape(-1).tolist(), 8, 2, 3)
    assert_plan_equal(got, info, ref)
    assert info["status"] & 1
    got, info, _ = run_plan(np.zeros((0, 4), np.int32), 8, 4, 1, dev=dev)
    assert info["n_chunks"] == 0 and info["total_rows"] == 0 and info["status"] == 0
    assert got["device_rows"] == [0, 0, 0, 0] and got["group_begin"] == [0] * 5


# ---------------------------------------------------------------------------
# permutation
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("T,K,E,P,hot", [(1, 1, 4, 2, 0.0), (700, 3, 12, 4, 0.7),
                                         (5000, 4, 64, 8, 0.9), (9000, 2, 8, 1, 0.5),
                                         (3000, 8, 16, 16, 0.0)])
def test_permutation_matches_oracle(dev, T, K, E, P, hot):
    import torch
    from paper_2601_17111_amd import binding as B
    rng = np.random.default_rng(T)
    ids = np.where(rng.random((T, K)) < hot, 1 % E, rng.integers(0, E, (T, K))).astype(np.int32)
    if T > 100:
        ids[5, 0] = E + 2  # one invalid id
    cap = math.ceil(T * K / P)
    _, info, (params, bufs, ids_t) = run_plan(ids, E, P, cap, dev=dev)
    D = 72
    x = torch.randn((T, D), device=dev, dtype=torch.float32).to(torch.bfloat16)
    gates = torch.rand((T, K), device=dev, dtype=torch.float32)
    R = T * K
    x_perm = torch.zeros((R, D), dtype=torch.bfloat16, device=dev)
    gate_perm = torch.zeros(R, dtype=torch.float32, device=dev)
    row_pair = torch.full((R,), -7, dtype=torch.int32, device=dev)
    pair_row = torch.zeros(R, dtype=torch.int32, device=dev)
    B.llep_permute(params, bufs, ids_t, gates, x, x_perm, gate_perm, row_pair, pair_row)
    torch.cuda.synchronize()
    ref = oracle.plan(ids.reshape(-1).tolist(), E, P, cap)
    pr_ref, rp_ref = oracle.permute(ids.reshape(-1).tolist(), ref, E)
    n = info["total_rows"]
    assert np.array_equal(pair_row.cpu().numpy(), pr_ref)
    assert np.array_equal(row_pair[:n].cpu().numpy(), rp_ref)
    rp = rp_ref.astype(np.int64)
    assert torch.equal(x_perm[:n].cpu(), x.cpu()[torch.from_numpy(rp // K)])
    assert torch.equal(gate_perm[:n].cpu(), gates.reshape(-1).cpu()[torch.from_numpy(rp)])


# ---------------------------------------------------------------------------
# whole layer
# ---------------------------------------------------------------------------

def _check_layer(run, tol, tokens=None):
    inp = run.inp
    cfg = run.cfg
    y = run.forward(-1).float().cpu().numpy()
    ref = oracle.plan(inp.ids.reshape(-1).tolist(), cfg.E, cfg.P, cfg.capacity, cfg.min_chunk,
                      lam=cfg.lam)
    info = run.layer.bufs.info_dict()
    b = run.layer.bufs
    nc, ng, nx = info["n_chunks"], info["n_groups"], info["n_xfers"]
    got = dict(
        loads=b.loads.cpu().tolist(),
        chunks=[tuple(c) for c in b.chunks[:nc].cpu().tolist()],
        chunk_row=b.chunk_row[:nc].cpu().tolist(),
        expert_chunk_begin=b.expert_chunk_begin.cpu().tolist(),
        groups=[tuple(g) for g in b.groups[:ng].cpu().tolist()],
        group_begin=b.group_begin.cpu().tolist(),
        device_rows=b.device_rows.cpu().tolist(),
        transfers=[tuple(x) for x in b.xfers[:nx].cpu().tolist()])
    assert_plan_equal(got, info, ref)
    pr_ref, rp_ref = oracle.permute(inp.ids.reshape(-1).tolist(), ref, cfg.E)
    assert np.array_equal(run.layer.pair_row.cpu().numpy(), pr_ref)
    W = run.host_weights(range(cfg.E))
    toks = list(range(cfg.T)) if tokens is None else tokens
    want = oracle.moe_output(inp.x, inp.ids, inp.gates, lambda e: W.get(e), toks)
    err = report(f"{cfg.name} y", y[toks], want)
    assert err <= tol, f"relative error {err:.3e} > {tol}"
    # out_perm rows against the per-row expert function
    rows = np.linspace(0, sum(ref.device_rows) - 1, num=min(64, sum(ref.device_rows))).astype(int)
    out = run.layer.out_perm.float().cpu().numpy()
    for r in rows:
        p = int(rp_ref[r])
        e = int(inp.ids.reshape(-1)[p])
        want_r = oracle.swiglu_ffn(inp.x[p // cfg.K][None, :], *W[e])[0]
        assert rel_err(out[r], want_r) <= tol
    return y


def test_tiny_fp32_layer(dev):
    from paper_2601_17111_amd.synth import CONFIGS
    run = LayerRun(CONFIGS["tiny-fp32"], 0, dev)
    _check_layer(run, TOL_F32)


@pytest.mark.parametrize("shape", [
    dict(T=1000, D=256, F=320, E=16, K=4, P=4),
    dict(T=777, D=128, F=192, E=8, K=2, P=8, distinct=False),
    dict(T=2048, D=512, F=128, E=32, K=8, P=8),
])
def test_bf16_layer_small(dev, shape):
    from fractions import Fraction
    from paper_2601_17111_amd.synth import LayerConfig
    cfg = LayerConfig("small-bf16", alpha=Fraction(11, 10), dtype="bf16",
                      routing=("hot", 0.7, 2), **shape)
    run = LayerRun(cfg, 3, dev)
    y_llep = _check_layer(run, TOL_BF16).copy()
    # LLEP does not change the layer's output: EP plan gives the same bits
    run.layer.set_mode("ep")
    y_ep = run.forward(-1).float().cpu().numpy()
    assert np.array_equal(y_llep, y_ep)
    # repeated runs are bit-identical
    run.layer.set_mode("llep")
    assert np.array_equal(run.forward(-1).float().cpu().numpy(), y_llep)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_pack_weights_layout(dev, dtype):
    """Every packed element sits where the header's block formula puts it."""
    import torch
    from paper_2601_17111_amd import binding as B
    E, D, F = 2, 128, 192
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    g = torch.Generator(device="cpu").manual_seed(3)
    wg, wu = (torch.randn(E, D, F, generator=g).to(tdt) for _ in range(2))
    wd = torch.randn(E, F, D, generator=g).to(tdt)
    gu, dn = B.llep_pack_weights(wg.to(dev), wu.to(dev), wd.to(dev))
    torch.cuda.synchronize()
    gu, dn = gu.cpu().reshape(E, -1), dn.cpu().reshape(E, -1)

    def idx(n, k, K):
        return ((n // 16) * (K // 32) + k // 32) * 512 + (n % 16) * 32 + k % 32

    n = np.arange(2 * F)[:, None]
    k = np.arange(D)[None, :]
    j, c = n // 64, n % 64
    col = 32 * j + c % 32
    for e in range(E):
        want = torch.where(torch.from_numpy(c < 32), wg[e].T[col[:, 0]], wu[e].T[col[:, 0]])
        assert torch.equal(gu[e][torch.from_numpy(idx(n, k, D))], want)
        nd = np.arange(D)[:, None]
        kf = np.arange(F)[None, :]
        assert torch.equal(dn[e][torch.from_numpy(idx(nd, kf, F))], wd[e].T)


def test_bf16_single_device_launch(dev):
    """llep_grouped_ffn on one device's groups writes exactly that device's rows."""
    import torch
    from fractions import Fraction
    from paper_2601_17111_amd.synth import LayerConfig
    cfg = LayerConfig("dev-bf16", T=1500, D=192, F=256, E=16, K=4, P=4, alpha=Fraction(11, 10),
                      dtype="bf16", routing=("hot", 0.8, 1))
    run = LayerRun(cfg, 1, dev)
    full = run.forward(-1)
    out_all = run.layer.out_perm.clone()
    info = run.layer.bufs.info_dict()
    rows = run.layer.bufs.device_rows.cpu().tolist()
    starts = np.concatenate([[0], np.cumsum(rows)])
    for d in range(cfg.P):
        run.layer.out_perm.fill_(float("nan"))
        run.layer.ffn(run.gu, run.dn, d)
        torch.cuda.synchronize()
        o = run.layer.out_perm[:info["total_rows"]]
        a, b = int(starts[d]), int(starts[d + 1])
        assert torch.equal(o[a:b], out_all[a:b])
        mask = torch.ones(info["total_rows"], dtype=torch.bool, device=o.device)
        mask[a:b] = False
        assert torch.isnan(o[mask].float()).all()
    del full


def test_empty_layer(dev):
    import torch
    from fractions import Fraction
    from paper_2601_17111_amd.synth import LayerConfig
    cfg = LayerConfig("empty", T=0, D=64, F=64, E=8, K=2, P=4, alpha=Fraction(1), dtype="bf16",
                      routing=("hot", 0.5, 1))
    from paper_2601_17111_amd import binding as B
    from paper_2601_17111_amd.layer import LLEPLayer
    layer = LLEPLayer(0, 2, 8, 4, 64, 64, 1, torch.bfloat16, dev)
    ids = torch.zeros((0, 2), dtype=torch.int32, device=dev)
    gates = torch.zeros((0, 2), dtype=torch.float32, device=dev)
    x = torch.zeros((0, 64), dtype=torch.bfloat16, device=dev)
    wg = torch.zeros((8, 64, 64), dtype=torch.bfloat16, device=dev)
    gu, dn = B.llep_pack_weights(wg, wg, wg)
    y = layer.forward(ids, gates, x, gu, dn, -1)
    torch.cuda.synchronize()
    assert y.shape == (0, 64) and layer.bufs.info_dict()["total_rows"] == 0
    del cfg


def test_bad_ids_skip_pairs_in_combine(dev):
    from fractions import Fraction
    from paper_2601_17111_amd.synth import LayerConfig
    cfg = LayerConfig("bad-ids", T=300, D=128, F=128, E=8, K=2, P=4, alpha=Fraction(5, 4),
                      dtype="f32", routing=("hot", 0.5, 1))
    run = LayerRun(cfg, 0, dev)
    ids = run.inp.ids.copy()
    ids[[3, 50, 299], [0, 1, 0]] = [8, -5, 100]
    run.inp.ids = ids
    import torch
    run.ids = torch.from_numpy(ids).to(dev)
    y = run.forward(-1).float().cpu().numpy()
    assert run.layer.bufs.info_dict()["status"] & 1
    W = run.host_weights(range(cfg.E))
    want = oracle.moe_output(run.inp.x, ids, run.inp.gates, lambda e: W.get(e))
    assert rel_err(y, want) <= TOL_F32
