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
