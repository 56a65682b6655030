"""llep_grouped_ffn_noalloc through the C ABI: the same expert outputs as
llep_grouped_ffn with a caller workspace (bit for bit, they share kernels),
on two calls in a row with the second on a smaller layer, for one device's
groups and for all devices; and a layer too large for the library's array is
rejected on the host."""

from fractions import Fraction

import numpy as np
import pytest

import oracle
from gpu_util import LayerRun, device, rel_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return device()


def _cfg(T, dtype):
    from paper_2601_17111_amd.synth import LayerConfig
    return LayerConfig(f"noalloc-{dtype}-T{T}", T=T, D=256, F=320, E=16, K=4, P=4,
                       alpha=Fraction(11, 10), dtype=dtype, routing=("hot", 0.7, 2))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_matches_caller_workspace(dev, dtype):
    import torch
    from paper_2601_17111_amd import binding as B
    for T in (900, 300):  # the second call is on a smaller layer
        run = LayerRun(_cfg(T, dtype), 1, dev)
        L = run.layer
        L.plan(run.ids)
        L.permute(run.ids, run.gates, run.x)
        info = L.bufs.info_dict()
        assert B.llep_grouped_ffn_workspace_bytes(L.params, run.cfg.F,
                                                  B.LLEP_BF16 if dtype == "bf16" else B.LLEP_F32
                                                  ) <= B.LLEP_NOALLOC_SCRATCH_BYTES
        for d in (info["max_device"], -1):  # all devices last: every row is then written
            L.out_perm.fill_(float("nan"))
            B.llep_grouped_ffn(L.params, L.bufs, d, L.x_perm, run.gu, run.dn, L.out_perm,
                               L.workspace)
            torch.cuda.synchronize()
            want = L.out_perm.clone()
            L.out_perm.fill_(float("nan"))
            B.llep_grouped_ffn_noalloc(L.params, L.bufs, d, L.x_perm, run.gu, run.dn,
                                       L.out_perm)
            torch.cuda.synchronize()
            assert torch.equal(torch.nan_to_num(L.out_perm, 7.0), torch.nan_to_num(want, 7.0)), \
                (T, d)
        # and a few rows against the oracle (the existing entry point's bar)
        n = info["total_rows"]
        rows = np.linspace(0, n - 1, 12).astype(int)
        row_pair = L.row_pair[:n].cpu().numpy()
        ids = run.inp.ids.reshape(-1)
        W = run.host_weights(range(run.cfg.E))
        got = L.out_perm[torch.from_numpy(rows).to(dev)].float().cpu().numpy()
        for i, r in enumerate(rows):
            p = int(row_pair[r])
            want_r = oracle.swiglu_ffn(run.inp.x[p // run.cfg.K][None], *W[int(ids[p])])[0]
            assert rel_err(got[i], want_r) <= (2e-2 if dtype == "bf16" else 1e-5)


def test_noalloc_rejects_layers_beyond_the_array(dev):
    import torch
    from paper_2601_17111_amd import binding as B
    from paper_2601_17111_amd.layer import LLEPLayer
    T, K, E, P, D, F = 16384, 8, 64, 8, 64, 2048  # (T K + 16 (2E + P)) F 2 bytes > 64 MiB
    params = B.make_params(T, K, E, P, T * K // P + 1)
    assert B.llep_grouped_ffn_workspace_bytes(params, F, B.LLEP_BF16) > \
        B.LLEP_NOALLOC_SCRATCH_BYTES
    layer = LLEPLayer(16, 1, 8, 4, D, 64, 4, torch.bfloat16, dev)  # buffers of a tiny layer
    x = torch.zeros((8, D), dtype=torch.bfloat16, device=dev)
    out = torch.zeros((8, D), dtype=torch.bfloat16, device=dev)
    w = torch.zeros(64 * D * F, dtype=torch.bfloat16, device=dev)
    with pytest.raises(B.LLEPError) as ei:
        B.llep_grouped_ffn_noalloc(params, layer.bufs, -1, x, w, w.reshape(64, D, F), out)
    assert ei.value.code == B.LLEP_E_WORKSPACE
    assert "LLEP_NOALLOC_SCRATCH_BYTES" in B.last_error()
