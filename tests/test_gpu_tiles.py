"""GPU parity of the grouped SwiGLU FFN at the edges of its tiling.

A group's rows are cut into m-tiles of 256 rows; its last m-tile is partly
filled unless the group's size is a multiple of 256. Every row of those
partly filled tiles is checked against the oracle (float64, Eq. 1 with the
SwiGLU expert of Sec. 5.1), for group sizes with every residue mod 256 that
changes which waves and which 32-row blocks of a tile hold valid rows, in
both projection kernels (256- and 192-column down-projection tiles), for the
inference and the training forward.

Also the same-work-over-more-experts shape of App. A.1 (65536 tokens, one
expert each, D = F = 8192, one device): first, middle and last row of every
group.
"""

from fractions import Fraction

import numpy as np
import pytest

import oracle
from gpu_util import LayerRun, device, rel_err, report

pytestmark = pytest.mark.gpu

TOL_BF16 = 2e-2

# residues mod 256 of the group sizes: one row, a 32-row block and its
# neighbours, the wave boundaries at 64 / 128 rows of a 2 x 4 wave layout,
# and a full tile less one row
RESIDUES = (1, 31, 32, 33, 63, 64, 65, 95, 96, 97, 127, 128, 129, 255)


@pytest.fixture(scope="module")
def dev():
    return device()


def _tile_cfg(D, F, base):
    from paper_2601_17111_amd.synth import LayerConfig
    loads = [base * (i % 2) + r for i, r in enumerate(RESIDUES)]
    E = len(loads)
    return LayerConfig(f"tiles-D{D}-F{F}", T=sum(loads), D=D, F=F, E=E, K=1, P=2,
                       alpha=Fraction(2), dtype="bf16", routing=("loads", tuple(loads)))


def _w64(W, e):
    return tuple(w.astype(np.float64) for w in W[e])


@pytest.mark.parametrize("D,F", [(2880, 2880), (2048, 768)], ids=["down192", "down256"])
def test_partial_mtiles_every_row(dev, D, F):
    import torch
    cfg = _tile_cfg(D, F, 256)
    run = LayerRun(cfg, 0, dev)
    L = run.layer
    run.forward(-1)
    out = L.out_perm.clone()
    info = L.bufs.info_dict()
    groups = L.bufs.groups[:info["n_groups"]].cpu().tolist()
    assert sorted(n % 256 for (_, _, _, n) in groups) == sorted(RESIDUES)
    row_pair = L.row_pair[:info["total_rows"]].cpu().numpy()
    W = run.host_weights(range(cfg.E))
    # the training forward writes the same expert outputs and keeps g, u
    L.ffn(run.gu, run.dn, -1, save_gate_up=True)
    torch.cuda.synchronize()
    assert torch.equal(L.out_perm, out)
    gu_saved = L.gate_up
    col = 32 * (np.arange(2 * F) // 64) + np.arange(2 * F) % 32
    is_gate = np.arange(2 * F) % 64 < 32
    worst = 0.0
    for (d, e, r0, n) in groups:
        first = r0 + (n - 1) // 256 * 256  # first row of the group's last m-tile
        rows = np.arange(first, r0 + n)
        rows_t = torch.from_numpy(rows).to(dev)
        wg, wu, wd = _w64(W, e)
        xr = run.inp.x[row_pair[rows]].astype(np.float64)
        want = oracle.swiglu_ffn(xr, wg, wu, wd)
        got = out[rows_t].float().cpu().numpy()
        for i, r in enumerate(rows):
            err = rel_err(got[i], want[i])
            worst = max(worst, err)
            assert err <= TOL_BF16, f"group ({d},{e}) n={n} row {r - r0} of the group: {err:.3e}"
        g = gu_saved[rows_t].float().cpu().numpy()
        want_gu = np.where(is_gate, (xr @ wg)[:, col], (xr @ wu)[:, col])
        for i in range(len(rows)):
            assert rel_err(g[i], want_gu[i]) <= TOL_BF16, (d, e, n, i)
    print(f"[{cfg.name}] worst per-row rel err of the partial m-tiles {worst:.3e}", flush=True)
    # one device's launch gives the same bits as the all-device launch
    starts = np.concatenate([[0], np.cumsum(L.bufs.device_rows.cpu().numpy())])
    for d in range(cfg.P):
        L.out_perm.zero_()
        L.ffn(run.gu, run.dn, d)
        torch.cuda.synchronize()
        a, b = int(starts[d]), int(starts[d + 1])
        assert torch.equal(L.out_perm[a:b], out[a:b])


@pytest.mark.slow
@pytest.mark.parametrize("N", [4, 64])
def test_a1_same_work_over_more_experts(dev, N):
    """App. A.1's shape: 65536 tokens, one expert each, spread evenly over N
    experts of one device, D = F = 8192; every group's first, middle and last
    row against the oracle."""
    import torch
    from paper_2601_17111_amd.synth import LayerConfig
    cfg = LayerConfig(f"a1-n{N}", T=65536, D=8192, F=8192, E=N, K=1, P=1,
                      alpha=Fraction(1), dtype="bf16", routing=("balanced",))
    run = LayerRun(cfg, 0, dev)
    run.forward(-1)
    L = run.layer
    info = L.bufs.info_dict()
    groups = L.bufs.groups[:info["n_groups"]].cpu().tolist()
    assert len(groups) == N and all(n == 65536 // N for (_, _, _, n) in groups)
    row_pair = L.row_pair[:info["total_rows"]].cpu().numpy()
    got_all, want_all = [], []
    for (d, e, r0, n) in groups:
        rows = np.array([r0, r0 + n // 2, r0 + n - 1])
        got = L.out_perm[torch.from_numpy(rows).to(dev)].float().cpu().numpy()
        w = tuple(t[e].cpu().double().numpy() for t in (run.wg, run.wu, run.wd))
        want = oracle.swiglu_ffn(run.inp.x[row_pair[rows]], *w)
        assert rel_err(got, want) <= TOL_BF16, (e, rel_err(got, want))
        got_all.append(got)
        want_all.append(want)
    report(cfg.name, np.concatenate(got_all), np.concatenate(want_all))


@pytest.mark.parametrize("D,F", [(2880, 2880), (2048, 768), (256, 320)],
                         ids=["down192", "down256", "small"])
def test_single_launch_waits_repeatable(dev, D, F):
    """Both projections run in one launch; a down-projection tile waits for
    the gate/up tiles of its rows, which may run on other XCDs. On a layer
    small enough that most workgroups start out waiting, twenty calls give
    the same bits, the LLEP and EP plans give the same bits per row, no wait
    gives up (status), and sampled rows match the oracle."""
    import torch
    from paper_2601_17111_amd import binding as B
    from paper_2601_17111_amd.synth import LayerConfig
    cfg = LayerConfig(f"wait-D{D}-F{F}", T=700, D=D, F=F, E=16, K=4, P=4,
                      alpha=Fraction(11, 10), dtype="bf16", routing=("hot", 0.8, 1))
    run = LayerRun(cfg, 2, dev)
    L = run.layer
    y0 = run.forward(-1).clone()
    out0 = L.out_perm.clone()
    for _ in range(20):
        L.ffn(run.gu, run.dn, -1)
        torch.cuda.synchronize()
        assert torch.equal(L.out_perm, out0)
    assert not L.bufs.info_dict()["status"] & B.LLEP_STATUS_FFN_WAIT
    L.set_mode("ep")
    assert torch.equal(run.forward(-1), y0)
    L.set_mode("llep")
    run.forward(-1)
    info = L.bufs.info_dict()
    n = info["total_rows"]
    rows = np.linspace(0, n - 1, 16).astype(int)
    row_pair = L.row_pair[:n].cpu().numpy()
    ids = run.inp.ids.reshape(-1)
    W = run.host_weights(range(cfg.E))
    got = L.out_perm[torch.from_numpy(rows).to(dev)].float().cpu().numpy()
    for i, r in enumerate(rows):
        p = int(row_pair[r])
        want = oracle.swiglu_ffn(run.inp.x[p // cfg.K][None], *_w64(W, int(ids[p])))[0]
        assert rel_err(got[i], want) <= TOL_BF16
