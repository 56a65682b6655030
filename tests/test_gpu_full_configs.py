"""GPU parity at the full sizes of the five layer shapes (and the gpt-oss-120b
hot-set sweep): plan and permutation bit-exact against the oracle; expert
outputs on sampled rows and tokens the oracle computes one by one; the
single-device launch the benchmark times."""

import numpy as np
import pytest

import oracle
from gpu_util import LayerRun, assert_plan_equal, device, rel_err, report

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

TOL_BF16 = 2e-2


@pytest.fixture(scope="module")
def dev():
    return device()


def _cfg(name):
    from paper_2601_17111_amd.synth import CONFIGS, gpt_oss_120b
    if name.startswith("gpt-oss-120b-hot"):
        return gpt_oss_120b(int(name[len("gpt-oss-120b-hot"):]))
    return CONFIGS[name]


PLAN_CASES = ([("tiny-fp32", 0), ("gpt-oss-20b", 0), ("qwen3-30b-a3b", 0), ("deepseek-v3", 0)] +
              [(f"gpt-oss-120b-hot{k}", s) for k in (16, 4, 1) for s in (0, 1, 2)])


@pytest.mark.parametrize("name,seed", PLAN_CASES, ids=lambda v: str(v))
def test_full_plan_and_permutation(dev, name, seed):
    import torch
    cfg = _cfg(name)
    run = LayerRun(cfg, seed, dev, weights=False)
    L = run.layer
    flat = run.inp.ids.reshape(-1).tolist()
    for mode in ("llep", "ep"):
        L.set_mode(mode)
        L.plan(run.ids)
        L.permute(run.ids, run.gates, run.x)
        torch.cuda.synchronize()
        ref = oracle.plan(flat, cfg.E, cfg.P, cfg.capacity, cfg.min_chunk, mode=mode)
        info = L.bufs.info_dict()
        nc, ng, nx = info["n_chunks"], info["n_groups"], info["n_xfers"]
        got = dict(
            loads=L.bufs.loads.cpu().tolist(),
            chunks=[tuple(c) for c in L.bufs.chunks[:nc].cpu().tolist()],
            chunk_row=L.bufs.chunk_row[:nc].cpu().tolist(),
            expert_chunk_begin=L.bufs.expert_chunk_begin.cpu().tolist(),
            groups=[tuple(g) for g in L.bufs.groups[:ng].cpu().tolist()],
            group_begin=L.bufs.group_begin.cpu().tolist(),
            device_rows=L.bufs.device_rows.cpu().tolist(),
            transfers=[tuple(x) for x in L.bufs.xfers[:nx].cpu().tolist()])
        assert_plan_equal(got, info, ref)
        if mode == "llep":
            # capacity holds (m = 1, P * cap >= R)
            assert max(ref.device_rows) <= cfg.capacity
        pr_ref, rp_ref = oracle.permute(flat, ref, cfg.E)
        assert np.array_equal(L.pair_row.cpu().numpy(), pr_ref)
        n = info["total_rows"]
        assert np.array_equal(L.row_pair[:n].cpu().numpy(), rp_ref)
        rp = torch.from_numpy(rp_ref.astype(np.int64))
        assert torch.equal(L.gate_perm[:n].cpu(), run.gates.reshape(-1).cpu()[rp])
        # x_perm rows: bit copies of their token rows (sampled)
        rng = np.random.default_rng(seed)
        rows = np.unique(np.concatenate([rng.integers(0, n, 2048), [0, n - 1]]))
        rows_t = torch.from_numpy(rows).to(dev)
        src = torch.from_numpy(rp_ref[rows] // cfg.K).to(dev)
        assert torch.equal(L.x_perm[rows_t], run.x[src])


# the paper's planner settings for its layer benchmarks (lambda = 1.3,
# alpha = 1, m = 1024) and the alpha / lambda ablation ranges, at full size
# (hot fraction on 4 experts, alpha, lambda, T, m); the last rows are chosen so
# the lambda bypass and the force-assign fire
KNOB_CASES = ([(frac, alpha, lam, T, 1024) for frac in (0.15, 0.3, 0.95)
               for alpha, lam, T in (("1", 1.3, 32768), ("2", 1.3, 32768), ("5/2", 2.6, 8192))] +
              [(0.05, "1", 2.6, 8192, 1024), (0.05, "1", 1.3, 8192, 1024),
               (0.3, "1", 1.3, 32768, 4096), (0.5, "1", 1.3, 8192, 2048)])


@pytest.mark.parametrize("frac,alpha,lam,T,m", KNOB_CASES, ids=lambda v: str(v))
def test_full_plan_paper_knobs(dev, frac, alpha, lam, T, m):
    """Plans with the min-chunk force-assign (m = 1024) and the lambda bypass
    active, bit-exact against the oracle; a bypassed plan is the EP plan."""
    from fractions import Fraction
    from paper_2601_17111_amd.synth import CONFIGS
    from gpu_util import run_plan
    cfg = CONFIGS["gpt-oss-120b"].with_(T=T, routing=("hot", frac, 4), alpha=Fraction(alpha),
                                        lam=lam, min_chunk=m)
    from paper_2601_17111_amd.synth import make_inputs
    ids = make_inputs(cfg, 0, with_x=False).ids
    got, info, _ = run_plan(ids, cfg.E, cfg.P, cfg.capacity, cfg.min_chunk, lam=cfg.lam, dev=dev)
    ref = oracle.plan(ids.reshape(-1).tolist(), cfg.E, cfg.P, cfg.capacity, cfg.min_chunk,
                      lam=cfg.lam)
    assert_plan_equal(got, info, ref)
    if ref.bypassed:
        ep = oracle.plan(ids.reshape(-1).tolist(), cfg.E, cfg.P, cfg.capacity, cfg.min_chunk,
                         mode="ep")
        assert ref.chunks == ep.chunks


def _expert_subset(cfg, ids, n_extra, rng):
    loads = np.bincount(ids.reshape(-1), minlength=cfg.E)
    order = np.argsort(-loads, kind="stable")
    hot = [int(e) for e in order[:max(1, n_extra // 2)]]
    rest = [int(e) for e in rng.permutation(order[len(hot):])[:n_extra - len(hot)]]
    return sorted(set(hot + rest))


FFN_CASES = [(n, 0) for n in ("gpt-oss-20b", "gpt-oss-120b-hot16", "gpt-oss-120b-hot4",
                               "gpt-oss-120b-hot1", "qwen3-30b-a3b", "deepseek-v3")]
FFN_CASES += [("gpt-oss-120b-hot1", 1), ("qwen3-30b-a3b", 2)]


@pytest.mark.parametrize("name,seed", FFN_CASES, ids=lambda v: str(v))
def test_full_layer_outputs(dev, name, seed):
    import torch
    cfg = _cfg(name)
    run = LayerRun(cfg, seed, dev)
    rng = np.random.default_rng(7 + seed)
    y = run.forward(-1).float().cpu().numpy()
    L = run.layer
    ids = run.inp.ids
    flat = ids.reshape(-1)
    S = _expert_subset(cfg, ids, 24 if cfg.E > 32 else cfg.E, rng)
    W = run.host_weights(S)
    info = L.bufs.info_dict()
    groups = L.bufs.groups[:info["n_groups"]].cpu().numpy()
    row_pair = L.row_pair[:info["total_rows"]].cpu().numpy()
    out = L.out_perm
    # rows of every group of a sampled expert: first, last and one inside
    checked = 0
    for (d, e, r0, n) in groups:
        if int(e) not in W:
            continue
        rows = sorted({int(r0), int(r0 + n - 1), int(r0 + rng.integers(0, n))})
        o = out[torch.tensor(rows, device=dev)].float().cpu().numpy()
        xs = run.inp.x[row_pair[rows] // cfg.K]
        want = oracle.swiglu_ffn(xs, *W[int(e)])
        err = rel_err(o, want)
        assert err <= TOL_BF16, f"group ({d},{e}) rows {rows}: {err:.3e}"
        checked += 1
    assert checked > 0
    # tokens whose experts are all sampled: boundary tokens first, then random
    ok_tok = np.all(np.isin(ids, S), axis=1)
    cand = np.nonzero(ok_tok)[0]
    assert len(cand) > 0
    chunks = L.bufs.chunks[:info["n_chunks"]].cpu().numpy()
    chunk_row = L.bufs.chunk_row[:info["n_chunks"]].cpu().numpy()
    boundary = set()
    for (d, e, s, t), r in zip(chunks, chunk_row):
        for rr in (int(r), int(r + t - s - 1)):
            tok = int(row_pair[rr]) // cfg.K
            if ok_tok[tok]:
                boundary.add(tok)
    sample = sorted(boundary)[:96]
    sample += [int(t) for t in rng.choice(cand, size=min(64, len(cand)), replace=False)]
    sample = sorted(set(sample))
    want = oracle.moe_output(run.inp.x, ids, run.inp.gates, lambda e: W.get(e), sample)
    err = report(f"{name} seed {seed} y", y[sample], want)
    assert err <= TOL_BF16, f"y relative error {err:.3e}"
    # the benchmark's launch: only the most loaded device's groups
    dstar = info["max_device"]
    starts = np.concatenate([[0], np.cumsum(L.bufs.device_rows.cpu().numpy())])
    a, b = int(starts[dstar]), int(starts[dstar + 1])
    ref_rows = out[a:b].clone()
    out[a:b].zero_()
    L.ffn(run.gu, run.dn, dstar)
    torch.cuda.synchronize()
    assert torch.equal(out[a:b], ref_rows)
    del flat


def test_full_ep_equals_llep_bitwise(dev):
    cfg = _cfg("gpt-oss-120b-hot1")
    run = LayerRun(cfg, 0, dev)
    y_llep = run.forward(-1).clone()
    assert run.layer.bufs.info_dict()["n_xfers"] > 0
    run.layer.set_mode("ep")
    y_ep = run.forward(-1)
    import torch
    assert torch.equal(y_llep, y_ep)


BWD_CASES = ["gpt-oss-20b", "gpt-oss-120b-hot1", "qwen3-30b-a3b", "deepseek-v3"]


@pytest.mark.parametrize("name", BWD_CASES)
def test_full_backward(dev, name):
    """Backward at full size: weight-gradient columns of sampled experts (the
    hot, spilled expert included) and input / gate gradients of sampled
    tokens against float64 gradients computed from the inputs; every
    device's partials summed in return order give the totals; under EP the
    input and gate gradients are the same bits."""
    import torch
    from paper_2601_17111_amd import binding as B
    cfg = _cfg(name)
    run = LayerRun(cfg, 0, dev)
    gut, dnt = B.llep_pack_weights_backward(run.wg, run.wu, run.wd)
    g = torch.Generator(device="cpu").manual_seed(11)
    dy_t = torch.randn(cfg.T, cfg.D, generator=g).to(torch.bfloat16)
    dy_dev = dy_t.to(dev)
    L = run.layer
    run.forward(-1)
    dx, dg, dwg, dwu, dwd = (t.clone() for t in L.backward(dy_dev, run.gates, run.gu, gut, dnt,
                                                          -1))
    torch.cuda.synchronize()
    assert L.bufs.info_dict()["n_xfers"] > 0 or name != "gpt-oss-120b-hot1"
    rng = np.random.default_rng(5)
    ids, gates = run.inp.ids, run.inp.gates
    S = _expert_subset(cfg, ids, 4, rng)
    W = run.host_weights(S)
    x = run.x.float().cpu().numpy().astype(np.float64)
    dy = dy_t.float().numpy().astype(np.float64)
    flat = ids.reshape(-1)
    # weight-gradient columns: all rows of expert e, plan-free
    for e in S:
        pairs = np.nonzero(flat == e)[0]
        if len(pairs) == 0:
            assert not dwg[e].any()
            continue
        wg, wu, wd = (w.astype(np.float64) for w in W[e])
        X = x[pairs // cfg.K]
        dO = gates.reshape(-1)[pairs, None].astype(np.float64) * dy[pairs // cfg.K]
        for f in rng.choice(cfg.F, size=2, replace=False):
            gc, uc = X @ wg[:, f], X @ wu[:, f]
            da = dO @ wd[f, :]
            s = 1.0 / (1.0 + np.exp(-gc))
            dgc = da * uc * s * (1 + gc * (1 - s))
            duc = da * gc * s
            for got, want in ((dwg[e][:, f], X.T @ dgc), (dwu[e][:, f], X.T @ duc),
                              (dwd[e][f, :], dO.T @ (gc * s * uc))):
                err = rel_err(got.cpu().numpy(), want)
                assert err <= TOL_BF16, (e, int(f), err)
    # input and gate gradients of tokens whose experts are all sampled
    ok_tok = np.nonzero(np.all(np.isin(ids, S), axis=1))[0]
    toks = rng.choice(ok_tok, size=min(24, len(ok_tok)), replace=False)
    dx_h = dx.float().cpu().numpy()
    dg_h = dg.cpu().numpy()
    dg_got, dg_want = [], []
    for t in toks:
        want_dx = np.zeros(cfg.D)
        for k in range(cfg.K):
            e = int(ids[t, k])
            wg, wu, wd = (w.astype(np.float64) for w in W[e])
            dv, _, _, _ = oracle.backward.swiglu_ffn_backward(x[t][None], wg, wu, wd,
                                                              gates[t, k] * dy[t][None])
            want_dx += dv[0]
            out = oracle.swiglu_ffn(x[t][None], wg, wu, wd)[0]
            dg_got.append(dg_h[t, k])
            dg_want.append(dy[t] @ out)
        assert rel_err(dx_h[t], want_dx) <= TOL_BF16, t
    # gate gradients of all sampled pairs (Eq. 1: d gate = dy . expert output),
    # against float64, under the same max-norm bound as every other output
    err = report(f"{name} d gates", np.array(dg_got), np.array(dg_want))
    assert err <= TOL_BF16, err
    # the gradient return: every device's partials, summed, give the totals
    acc = [torch.zeros_like(w) for w in (dwg, dwu, dwd)]
    for d in range(cfg.P):
        parts = L.backward(dy_dev, run.gates, run.gu, gut, dnt, d)[2:]
        for a, p in zip(acc, parts):
            a += p
    torch.cuda.synchronize()
    for a, tot in zip(acc, (dwg, dwu, dwd)):
        den = tot.abs().max().item()
        assert (a - tot).abs().max().item() <= 1e-5 * den
    del acc
    # training forward: the backward from the saved gate / up values gives
    # the same bits as the one that recomputes them
    L.forward(run.ids, run.gates, run.x, run.gu, run.dn, -1, save_gate_up=True)
    saved = L.backward(dy_dev, run.gates, run.gu, gut, dnt, -1)
    torch.cuda.synchronize()
    for a, b in zip(saved, (dx, dg, dwg, dwu, dwd)):
        assert torch.equal(a, b)
    del saved
    # the saved g, u themselves: sampled rows of the sampled experts' groups
    # against the float64 projections of their token rows
    info = L.bufs.info_dict()
    row_pair = L.row_pair[:info["total_rows"]].cpu().numpy()
    col = 32 * (np.arange(2 * cfg.F) // 64) + np.arange(2 * cfg.F) % 32
    is_gate = np.arange(2 * cfg.F) % 64 < 32
    checked = 0
    for (d, e, r0, n) in L.bufs.groups[:info["n_groups"]].cpu().tolist():
        if e not in S:
            continue
        rows = np.unique(np.array([r0, r0 + n - 1, r0 + int(rng.integers(0, n))]))
        got = L.gate_up[torch.from_numpy(rows).to(dev)].float().cpu().numpy()
        wg, wu, _ = (w.astype(np.float64) for w in W[e])
        xr = x[row_pair[rows] // cfg.K]
        want = np.where(is_gate, (xr @ wg)[:, col], (xr @ wu)[:, col])
        assert rel_err(got, want) <= TOL_BF16, (d, e)
        checked += 1
    assert checked > 0
    L.gate_up = None
    if name != "deepseek-v3":
        L.set_mode("ep")
        run.forward(-1)
        dx_ep, dg_ep, dwg_ep = (t.clone() for t in L.backward(dy_dev, run.gates, run.gu, gut,
                                                              dnt, -1)[:3])
        torch.cuda.synchronize()
        assert torch.equal(dx_ep, dx)
        assert torch.equal(dg_ep, dg)
        assert (dwg_ep - dwg).abs().max().item() <= 1e-5 * dwg.abs().max().item()
