"""GPU parity of the backward pass against the oracle: the combine's backward
exactly (up to float32 summation order), the layer's input, gate and weight
gradients within the bf16 tolerance, the per-device partial weight gradients
and the gradient return, and the edge cases."""

import numpy as np
import pytest

import oracle
from gpu_util import LayerRun, device, rel_err

pytestmark = pytest.mark.gpu

TOL_BF16 = 2e-2
TOL_F32 = 1e-5


@pytest.fixture(scope="module")
def dev():
    return device()


def _cfg(name, alpha=(11, 10), routing=("hot", 0.7, 2), **shape):
    from fractions import Fraction
    from paper_2601_17111_amd.synth import LayerConfig
    return LayerConfig(name, alpha=Fraction(*alpha), dtype="bf16", routing=routing, **shape)


def _dy(cfg, seed, dev):
    import torch
    g = torch.Generator(device="cpu").manual_seed(1000 + seed)
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    return torch.randn(cfg.T, cfg.D, generator=g).to(dt).to(dev)


class BwdRun(LayerRun):
    def __init__(self, cfg, seed, dev, mode="llep"):
        super().__init__(cfg, seed, dev, mode)
        import torch
        from paper_2601_17111_amd import binding as B
        self.gut, self.dnt = B.llep_pack_weights_backward(self.wg, self.wu, self.wd)
        self.dy = _dy(cfg, seed, dev)
        torch.cuda.synchronize()

    def backward(self, device=-1, save=False, fwd_device=-1):
        """save: training forward (g and u kept) over fwd_device's groups."""
        import torch
        self.layer.forward(self.ids, self.gates, self.x, self.gu, self.dn, fwd_device,
                           save_gate_up=save)
        out = self.layer.backward(self.dy, self.gates, self.gu, self.gut, self.dnt, device)
        torch.cuda.synchronize()
        return [t.float().cpu().numpy() for t in out]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_pack_weights_backward_layout(dev, dtype):
    """Every element of the backward packing sits where the header puts it."""
    import torch
    from paper_2601_17111_amd import binding as B
    E, D, F = 2, 128, 192
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    g = torch.Generator(device="cpu").manual_seed(5)
    wg, wu = (torch.randn(E, D, F, generator=g).to(tdt) for _ in range(2))
    wd = torch.randn(E, F, D, generator=g).to(tdt)
    gut, dnt = B.llep_pack_weights_backward(wg.to(dev), wu.to(dev), wd.to(dev))
    torch.cuda.synchronize()
    gut, dnt = gut.cpu().reshape(E, -1), dnt.cpu().reshape(E, -1)

    def idx(n, k, K):
        return ((n // 16) * (K // 32) + k // 32) * 512 + (n % 16) * 32 + k % 32

    n = np.arange(D)[:, None]
    k = np.arange(2 * F)[None, :]
    col = 32 * (k // 64) + k % 32
    for e in range(E):
        want = torch.where(torch.from_numpy(np.broadcast_to(k % 64 < 32, (D, 2 * F))),
                           wg[e][:, col[0]], wu[e][:, col[0]])
        assert torch.equal(gut[e][torch.from_numpy(idx(n, k, 2 * F))], want)
        nf = np.arange(F)[:, None]
        kd = np.arange(D)[None, :]
        assert torch.equal(dnt[e][torch.from_numpy(idx(nf, kd, D))], wd[e])


def test_combine_backward_rows_and_gates(dev):
    """d_out_perm = gate * dy with one rounding (bit-exact); d gates are the
    dot products of dy with the expert rows the forward produced."""
    import torch
    cfg = _cfg("cb", T=613, D=192, F=128, E=8, K=3, P=4)
    run = BwdRun(cfg, 2, dev)
    run.backward(-1)
    L = run.layer
    pr = L.pair_row.cpu().numpy()[:cfg.T * cfg.K]
    want_rows = (run.gates.reshape(-1, 1).cpu() * run.dy.float().cpu().repeat_interleave(cfg.K, 0)
                 ).to(torch.bfloat16)
    got_rows = L.d_out_perm.cpu()[torch.from_numpy(pr.astype(np.int64))]
    assert torch.equal(got_rows, want_rows)
    out = L.out_perm.float().cpu().numpy().astype(np.float64)[pr]
    dy = run.dy.float().cpu().numpy().astype(np.float64)
    want_g = np.einsum("pd,pd->p", np.repeat(dy, cfg.K, 0), out).reshape(cfg.T, cfg.K)
    got_g = L.d_gates.cpu().numpy()
    assert np.allclose(got_g, want_g, rtol=1e-5, atol=1e-5 * np.abs(want_g).max())


@pytest.mark.parametrize("T,K,D,dtype", [(37, 70, 4096, "bf16"), (200, 5, 136, "bf16"),
                                         (3, 4, 8, "bf16"), (50, 4, 2560, "bf16"),
                                         (41, 6, 2880, "bf16"), (37, 70, 2048, "f32"),
                                         (200, 5, 72, "f32"), (3, 4, 8, "f32")])
def test_combine_backward_standalone(dev, T, K, D, dtype):
    """Rows longer than one wave slice, rows of a ragged number of vectors,
    K > 64 (two 64-pair batches), and an invalid pair; bf16 and float32."""
    import torch
    from paper_2601_17111_amd import binding as B
    E, P = 8, 2
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    rng = np.random.default_rng(9 + D)
    ids = rng.integers(0, E, (T, K)).astype(np.int32)
    ids[min(5, T - 1), 3] = E + 1  # an invalid pair: no row, d gate 0
    params = B.make_params(T, K, E, P, T * K)
    bufs = B.PlanBuffers(params, dev)
    ids_t = torch.from_numpy(ids).to(dev)
    gates = torch.from_numpy(rng.random((T, K)).astype(np.float32)).to(dev)
    x = torch.randn(T, D, device=dev).to(tdt)
    R = T * K
    x_perm = torch.empty(R, D, dtype=tdt, device=dev)
    gp = torch.empty(R, dtype=torch.float32, device=dev)
    rp = torch.empty(R, dtype=torch.int32, device=dev)
    pr = torch.empty(R, dtype=torch.int32, device=dev)
    B.llep_plan(params, ids_t, bufs)
    B.llep_permute(params, bufs, ids_t, gates, x, x_perm, gp, rp, pr)
    out_perm = torch.randn(R, D, device=dev).to(tdt)
    dy = torch.randn(T, D, device=dev).to(tdt)
    d_out = torch.zeros(R, D, dtype=tdt, device=dev)
    dg = torch.full((T, K), 7.0, device=dev)
    B.llep_combine_backward(params, out_perm, pr, gates, dy, d_out, dg)
    torch.cuda.synchronize()
    prn = pr.cpu().numpy()
    bad = min(5, T - 1) * K + 3
    assert prn[bad] == -1
    valid = prn >= 0
    o = out_perm.float().cpu().numpy().astype(np.float64)
    d = dy.float().cpu().numpy().astype(np.float64)
    want = np.zeros(R)
    want[valid] = np.einsum("pd,pd->p", np.repeat(d, K, 0)[valid], o[prn[valid]])
    got = dg.cpu().numpy().reshape(-1)
    assert got[bad] == 0.0
    assert np.allclose(got, want, rtol=1e-5, atol=1e-5 * np.abs(want).max())
    g = gates.cpu().numpy().reshape(-1)
    want_rows = (torch.from_numpy(g[valid]).reshape(-1, 1) *
                 torch.from_numpy(np.repeat(d, K, 0)[valid]).float()).to(tdt)
    assert torch.equal(d_out.cpu()[torch.from_numpy(prn[valid].astype(np.int64))], want_rows)


SHAPES = [
    dict(T=1000, D=256, F=320, E=16, K=4, P=4),
    dict(T=777, D=128, F=192, E=8, K=2, P=8),
    dict(T=600, D=192, F=256, E=12, K=3, P=4),
    dict(T=97, D=64, F=64, E=4, K=1, P=2),
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"T{s['T']}D{s['D']}F{s['F']}E{s['E']}")
@pytest.mark.parametrize("mode", ["llep", "ep"])
def test_layer_backward_matches_oracle(dev, shape, mode):
    """dx, d gates and the per-expert weight gradients (after the gradient
    return) against the plan-free gradients of the oracle."""
    cfg = _cfg("bwd", **shape)
    run = BwdRun(cfg, 4, dev, mode)
    dx, dgates, dwg, dwu, dwd = run.backward(-1)
    W = run.host_weights(range(cfg.E))
    dy = run.dy.float().cpu().numpy()
    x = run.x.float().cpu().numpy()
    want_dx, want_dg, want_dW = oracle.moe_backward(x, run.inp.ids, run.inp.gates,
                                                    lambda e: W[e], dy, cfg.E)
    assert rel_err(dx, want_dx) <= TOL_BF16
    assert rel_err(dgates, want_dg) <= TOL_BF16
    for e in range(cfg.E):
        if e not in want_dW:
            assert not dwg[e].any() and not dwu[e].any() and not dwd[e].any()
            continue
        for got, want in zip((dwg[e], dwu[e], dwd[e]), want_dW[e]):
            assert rel_err(got, want) <= TOL_BF16, e


def test_backward_llep_equals_ep_per_row(dev):
    """The input and gate gradients are row-local: the LLEP and EP plans give
    the same bits; the weight gradients agree up to summation order."""
    cfg = _cfg("bwd-eq", T=900, D=128, F=192, E=8, K=4, P=4, routing=("hot", 0.8, 1))
    a = BwdRun(cfg, 6, dev, "llep").backward(-1)
    b = BwdRun(cfg, 6, dev, "ep").backward(-1)
    assert np.array_equal(a[0], b[0])
    assert np.array_equal(a[1], b[1])
    for x, y in zip(a[2:], b[2:]):
        assert rel_err(x, y) <= 1e-5


def test_backward_device_partials_and_return(dev):
    """Per device: its partial weight gradients equal the oracle's partials of
    that device's groups, only its experts are written, only its rows of
    dx_perm are written; the partials added in return order give the totals."""
    import torch
    cfg = _cfg("bwd-dev", T=1500, D=192, F=256, E=16, K=4, P=4, routing=("hot", 0.8, 1))
    run = BwdRun(cfg, 1, dev)
    tot = [t.copy() for t in run.backward(-1)[2:]]
    L = run.layer
    dx_perm_all = L.dx_perm.clone()
    ids_flat = run.inp.ids.reshape(-1)
    pl = oracle.plan(ids_flat.tolist(), cfg.E, cfg.P, cfg.capacity, cfg.min_chunk, lam=cfg.lam)
    _, row_pair = oracle.permute(ids_flat.tolist(), pl, cfg.E)
    W = run.host_weights(range(cfg.E))
    x = run.x.float().cpu().numpy()
    dy = run.dy.float().cpu().numpy()
    _, partials, dW = oracle.plan_backward(x, ids_flat, run.inp.gates.reshape(-1), lambda e: W[e],
                                           dy, pl, np.asarray(row_pair), cfg.K, cfg.E // cfg.P)
    assert any(d != e // (cfg.E // cfg.P) for (d, e) in partials)  # something spilled
    rows = L.bufs.device_rows.cpu().tolist()
    starts = np.concatenate([[0], np.cumsum(rows)])
    summed = {}
    M = cfg.E // cfg.P
    for d in range(cfg.P):
        L.dx_perm.fill_(float("nan"))
        parts = [t.copy() for t in run.backward(d)[2:]]
        dxp = L.dx_perm[:int(starts[-1])]
        a, b = int(starts[d]), int(starts[d + 1])
        assert torch.equal(dxp[a:b], dx_perm_all[a:b])
        mask = torch.ones(dxp.shape[0], dtype=torch.bool, device=dxp.device)
        mask[a:b] = False
        assert torch.isnan(dxp[mask].float()).all()
        mine = {e for (dd, e) in partials if dd == d}
        for e in range(cfg.E):
            if e not in mine:
                assert not any(p[e].any() for p in parts)
                continue
            for got, want in zip((p[e] for p in parts), partials[(d, e)]):
                assert rel_err(got, want) <= TOL_BF16, (d, e)
            summed.setdefault(e, []).append((d, [p[e].astype(np.float64) for p in parts]))
    for e, lst in summed.items():
        lst.sort(key=lambda t: (t[0] != e // M, t[0]))  # native first, then by device
        acc = [np.zeros_like(q) for q in lst[0][1]]
        for _, ps in lst:
            acc = [u + v for u, v in zip(acc, ps)]
        for s, t, want in zip(acc, (tot[0][e], tot[1][e], tot[2][e]), dW[e]):
            assert rel_err(t, s) <= 1e-5, e
            assert rel_err(t, want) <= TOL_BF16, e


def test_backward_empty_and_single_rows(dev):
    """T == 0 enqueues nothing; groups of one row (every expert hit once)."""
    import torch
    from paper_2601_17111_amd import binding as B
    from paper_2601_17111_amd.layer import LLEPLayer
    layer = LLEPLayer(0, 2, 8, 4, 64, 64, 1, torch.bfloat16, dev)
    z = torch.zeros((8, 64, 64), dtype=torch.bfloat16, device=dev)
    gu, dn = B.llep_pack_weights(z, z, z)
    gut, dnt = B.llep_pack_weights_backward(z, z, z)
    ids = torch.zeros((0, 2), dtype=torch.int32, device=dev)
    gates = torch.zeros((0, 2), dtype=torch.float32, device=dev)
    x = torch.zeros((0, 64), dtype=torch.bfloat16, device=dev)
    layer.forward(ids, gates, x, gu, dn, -1)
    out = layer.backward(torch.zeros((0, 64), dtype=torch.bfloat16, device=dev), gates, gu, gut,
                         dnt, -1)
    torch.cuda.synchronize()
    assert out[0].shape == (0, 64)
    assert not any(t.any() for t in out[2:])
    # one pair per expert: groups of a single row
    cfg = _cfg("bwd-one", T=8, D=64, F=128, E=8, K=1, P=2, routing=("hot", 0.0, 1))
    run = BwdRun(cfg, 0, dev)
    ids1 = np.arange(8, dtype=np.int32).reshape(8, 1)
    run.inp.ids = ids1
    run.ids = torch.from_numpy(ids1).to(dev)
    dx, dgates, dwg, dwu, dwd = run.backward(-1)
    W = run.host_weights(range(cfg.E))
    want_dx, want_dg, want_dW = oracle.moe_backward(run.x.float().cpu().numpy(), ids1,
                                                    run.inp.gates, lambda e: W[e],
                                                    run.dy.float().cpu().numpy(), cfg.E)
    assert rel_err(dx, want_dx) <= TOL_BF16
    assert rel_err(dgates, want_dg) <= TOL_BF16
    for e in range(cfg.E):
        for got, want in zip((dwg[e], dwu[e], dwd[e]), want_dW[e]):
            assert rel_err(got, want) <= TOL_BF16, e


def test_backward_rejects_bad_arguments(dev):
    import ctypes
    from paper_2601_17111_amd import binding as B
    params = B.make_params(16, 2, 8, 4, 8)
    assert B.llep_grouped_ffn_backward_workspace_bytes(params, 64, 64, 7) == 0
    assert B.llep_grouped_ffn_backward_workspace_bytes(params, 64, 64, B.LLEP_BF16) > 0
    a = ctypes.c_void_p(4096)
    assert B.lib().llep_pack_weights_backward(8, 64, 64, 7, a, a, a, a, a, None) == B.LLEP_E_DTYPE


def test_f32_backward_tiny_layer(dev):
    """The float32 path on the tiny layer: input, gate and weight gradients
    against the plan-free float64 gradients, and every device's partials
    against the oracle's partials of the same plan, to 1e-5."""
    from paper_2601_17111_amd.synth import CONFIGS
    cfg = CONFIGS["tiny-fp32"]
    run = BwdRun(cfg, 0, dev)
    tot = [t.copy() for t in run.backward(-1)]
    ids_flat = run.inp.ids.reshape(-1)
    pl = oracle.plan(ids_flat.tolist(), cfg.E, cfg.P, cfg.capacity, cfg.min_chunk, lam=cfg.lam)
    assert any(d != e // (cfg.E // cfg.P) for (d, e, _, _) in pl.groups)  # spilled chunks
    _, row_pair = oracle.permute(ids_flat.tolist(), pl, cfg.E)
    W = run.host_weights(range(cfg.E))
    x = run.x.cpu().numpy()
    dy = run.dy.cpu().numpy()
    _, partials, dW = oracle.plan_backward(x, ids_flat, run.inp.gates.reshape(-1), lambda e: W[e],
                                           dy, pl, np.asarray(row_pair), cfg.K, cfg.E // cfg.P)
    want_dx, want_dg, want_dW = oracle.moe_backward(x, run.inp.ids, run.inp.gates,
                                                    lambda e: W[e], dy, cfg.E)
    assert rel_err(tot[0], want_dx) <= TOL_F32
    assert rel_err(tot[1], want_dg) <= TOL_F32
    for e in range(cfg.E):
        for got, want in zip((tot[2][e], tot[3][e], tot[4][e]), want_dW[e]):
            assert rel_err(got, want) <= TOL_F32, e
    for d in range(cfg.P):
        parts = run.backward(d)[2:]
        for (dd, e), want in partials.items():
            if dd != d:
                continue
            for got, w in zip((p[e] for p in parts), want):
                assert rel_err(got, w) <= TOL_F32, (d, e)


def test_backward_force_assign_plan(dev):
    """A plan where Alg. 3 force-assigns (min chunk 150 under capacity
    ceil(R / P)): per-device partials against the oracle's partials of the
    same plan, and the totals against the plan-free gradients."""
    cfg = _cfg("bwd-force", alpha=(1, 1), routing=("hot", 0.5, 3), T=700, D=128, F=192, E=8,
               K=3, P=4).with_(min_chunk=150)
    run = BwdRun(cfg, 9, dev)
    tot = [t.copy() for t in run.backward(-1)]
    ids_flat = run.inp.ids.reshape(-1)
    pl = oracle.plan(ids_flat.tolist(), cfg.E, cfg.P, cfg.capacity, cfg.min_chunk, lam=cfg.lam)
    assert pl.forced > 0
    assert run.layer.bufs.info_dict()["forced"] == pl.forced
    assert run.layer.bufs.groups[:len(pl.groups)].cpu().tolist() == [list(g) for g in pl.groups]
    _, row_pair = oracle.permute(ids_flat.tolist(), pl, cfg.E)
    W = run.host_weights(range(cfg.E))
    x = run.x.float().cpu().numpy()
    dy = run.dy.float().cpu().numpy()
    _, partials, dW = oracle.plan_backward(x, ids_flat, run.inp.gates.reshape(-1), lambda e: W[e],
                                           dy, pl, np.asarray(row_pair), cfg.K, cfg.E // cfg.P)
    want_dx, want_dg, _ = oracle.moe_backward(x, run.inp.ids, run.inp.gates, lambda e: W[e], dy,
                                              cfg.E)
    assert rel_err(tot[0], want_dx) <= TOL_BF16
    assert rel_err(tot[1], want_dg) <= TOL_BF16
    for e, want in dW.items():
        for got, w in zip((tot[2][e], tot[3][e], tot[4][e]), want):
            assert rel_err(got, w) <= TOL_BF16, e
    for d in range(cfg.P):
        parts = run.backward(d)[2:]
        for (dd, e), want in partials.items():
            if dd != d:
                continue
            for got, w in zip((p[e] for p in parts), want):
                assert rel_err(got, w) <= TOL_BF16, (d, e)


def test_backward_with_invalid_ids(dev):
    """Pairs routed to an id outside [0, E) contribute nothing to any
    gradient and get a zero gate gradient, as in the plan-free definition."""
    import torch
    cfg = _cfg("bwd-bad", T=300, D=128, F=128, E=8, K=2, P=4, routing=("hot", 0.5, 1))
    run = BwdRun(cfg, 0, dev)
    ids = run.inp.ids.copy()
    ids[[3, 50, 299], [0, 1, 0]] = [8, -5, 100]
    run.inp.ids = ids
    run.ids = torch.from_numpy(ids).to(dev)
    dx, dgates, dwg, dwu, dwd = run.backward(-1)
    assert run.layer.bufs.info_dict()["status"] & 1
    W = run.host_weights(range(cfg.E))
    want_dx, want_dg, want_dW = oracle.moe_backward(run.x.float().cpu().numpy(), ids, run.inp.gates,
                                                    lambda e: W[e], run.dy.float().cpu().numpy(),
                                                    cfg.E)
    assert rel_err(dx, want_dx) <= TOL_BF16
    assert rel_err(dgates, want_dg) <= TOL_BF16
    assert dgates[3, 0] == 0.0 and dgates[50, 1] == 0.0 and dgates[299, 0] == 0.0
    for e, want in want_dW.items():
        for got, w in zip((dwg[e], dwu[e], dwd[e]), want):
            assert rel_err(got, w) <= TOL_BF16, e


@pytest.mark.parametrize("shape", SHAPES[:3] + ["tiny-fp32"],
                         ids=lambda s: s if isinstance(s, str) else
                         f"T{s['T']}D{s['D']}F{s['F']}E{s['E']}")
def test_train_forward_saves_gate_up(dev, shape):
    """The training forward gives the inference forward's bits and stores g
    and u of exactly the rows of its device range, each within the dtype's
    tolerance of the float64 projections."""
    import torch
    from paper_2601_17111_amd.synth import CONFIGS
    cfg = CONFIGS[shape] if isinstance(shape, str) else _cfg("train-fwd", **shape)
    tol = TOL_BF16 if cfg.dtype == "bf16" else TOL_F32
    run = BwdRun(cfg, 3, dev)
    L = run.layer
    run.forward(-1)
    out_ref, y_ref = L.out_perm.clone(), L.y.clone()
    L.gate_up = torch.full((cfg.T * cfg.K, 2 * cfg.F), float("nan"), dtype=run.tdt, device=dev)
    L.forward(run.ids, run.gates, run.x, run.gu, run.dn, -1, save_gate_up=True)
    torch.cuda.synchronize()
    total = int(L.bufs.device_rows.sum().item())
    assert torch.equal(L.out_perm[:total], out_ref[:total])
    assert torch.equal(L.y, y_ref)
    gu = L.gate_up[:total].float().cpu().numpy()
    assert np.isfinite(gu).all()
    xp = L.x_perm[:total].float().cpu().numpy().astype(np.float64)
    W = run.host_weights(range(cfg.E))
    rows_expert = np.full(total, -1)
    ng = L.bufs.info_dict()["n_groups"]
    for (d, e, r0, n) in L.bufs.groups[:ng].cpu().tolist():
        rows_expert[r0:r0 + n] = e
    col = 32 * (np.arange(2 * cfg.F) // 64) + np.arange(2 * cfg.F) % 32
    is_gate = np.arange(2 * cfg.F) % 64 < 32
    for e in range(cfg.E):
        rows = np.nonzero(rows_expert == e)[0]
        if len(rows) == 0:
            continue
        wg, wu, _ = (w.astype(np.float64) for w in W[e])
        want = np.where(is_gate, (xp[rows] @ wg)[:, col], (xp[rows] @ wu)[:, col])
        assert rel_err(gu[rows], want) <= tol, e
    # one device's range: only its rows are written
    rows = L.bufs.device_rows.cpu().tolist()
    starts = np.concatenate([[0], np.cumsum(rows)])
    d = int(np.argmax(rows))
    L.gate_up.fill_(float("nan"))
    L.forward(run.ids, run.gates, run.x, run.gu, run.dn, d, save_gate_up=True)
    torch.cuda.synchronize()
    a, b = int(starts[d]), int(starts[d + 1])
    g2 = L.gate_up.float()
    assert torch.isfinite(g2[a:b]).all()
    assert torch.isnan(g2[:a]).all() and torch.isnan(g2[b:]).all()
    assert np.array_equal(g2[a:b].cpu().numpy(), gu[a:b])


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_backward_from_saved_gate_up_is_bit_identical(dev, dtype):
    """Backward from the training forward's g and u equals the backward that
    recomputes them, bit for bit, for the whole layer and for one device's
    range (saved by a forward over all devices or over that device)."""
    from paper_2601_17111_amd.synth import CONFIGS
    if dtype == "bf16":
        cfg = _cfg("saved-gu", T=1000, D=256, F=320, E=16, K=4, P=4)
    else:
        cfg = CONFIGS["tiny-fp32"]
    run = BwdRun(cfg, 8, dev)
    ref = run.backward(-1)
    got = run.backward(-1, save=True)
    for a, b in zip(got, ref):
        assert np.array_equal(a, b)
    d = 1
    ref_d = run.backward(d)
    for fwd in (-1, d):
        got_d = run.backward(d, save=True, fwd_device=fwd)
        for a, b in zip(got_d[2:], ref_d[2:]):
            assert np.array_equal(a, b), fwd


@pytest.mark.parametrize("E,P,alpha", [(512, 64, (1, 1)), (512, 8, (11, 10)), (256, 64, (5, 4))])
def test_layer_max_experts_and_devices(dev, E, P, alpha):
    """The largest expert and device counts the library takes (512 experts,
    64 devices), zipf routing with many spills: the layer output, the input
    and gate gradients and every expert's weight gradients against the
    oracle's plan-free values, and every device's partials summed in return
    order give the totals."""
    import torch
    cfg = _cfg("max", alpha=alpha, routing=("zipf", 1.2), T=1500, D=64, F=64, E=E, K=8, P=P)
    run = BwdRun(cfg, 12, dev)
    y = run.forward(-1).float().cpu().numpy()
    W = run.host_weights(range(E))
    x = run.x.float().cpu().numpy()
    want_y = oracle.moe_output(x, run.inp.ids, run.inp.gates, lambda e: W[e])
    assert rel_err(y, want_y) <= TOL_BF16
    dx, dgates, dwg, dwu, dwd = run.backward(-1, save=True)
    assert run.layer.bufs.info_dict()["n_xfers"] > 0
    want_dx, want_dg, want_dW = oracle.moe_backward(x, run.inp.ids, run.inp.gates,
                                                    lambda e: W[e], run.dy.float().cpu().numpy(),
                                                    E)
    assert rel_err(dx, want_dx) <= TOL_BF16
    assert rel_err(dgates, want_dg) <= TOL_BF16
    for e in range(E):
        if e not in want_dW:
            assert not dwg[e].any() and not dwd[e].any()
            continue
        for got, want in zip((dwg[e], dwu[e], dwd[e]), want_dW[e]):
            assert rel_err(got, want) <= TOL_BF16, e
    acc = [np.zeros_like(t) for t in (dwg, dwu, dwd)]
    for d in range(P):
        for a, p in zip(acc, run.backward(d)[2:]):
            a += p
    for a, t in zip(acc, (dwg, dwu, dwd)):
        assert rel_err(a, t) <= 1e-5
