"""Helpers for the GPU parity tests: run the library through its binding on
seeded inputs and compare with the oracle."""

from __future__ import annotations

import numpy as np

import oracle


def device():
    import pytest
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2601_17111_amd import binding as B
    B.lib()  # raises when the library is missing: no fallback
    return "cuda:0"


def run_plan(ids_np: np.ndarray, E: int, P: int, cap: int, m: int = 1, mode: str = "llep",
             lam: float = 0.0, dev: str = "cuda:0"):
    """llep_plan on the GPU; returns (tables as numpy, info dict, layer bufs)."""
    import torch
    from paper_2601_17111_amd import binding as B
    ids2 = ids_np if ids_np.ndim == 2 else ids_np.reshape(-1, 1)
    ids2 = np.ascontiguousarray(ids2.astype(np.int32))
    T, K = ids2.shape
    params = B.make_params(T, K, E, P, cap, m, lam, mode)
    bufs = B.PlanBuffers(params, dev)
    ids_t = torch.from_numpy(ids2).to(dev)
    B.llep_plan(params, ids_t, bufs)
    torch.cuda.synchronize()
    info = bufs.info_dict()
    nc, ng, nx = info["n_chunks"], info["n_groups"], info["n_xfers"]
    tables = dict(
        loads=bufs.loads.cpu().tolist(),
        chunks=[tuple(c) for c in bufs.chunks[:nc].cpu().tolist()],
        chunk_row=bufs.chunk_row[:nc].cpu().tolist(),
        expert_chunk_begin=bufs.expert_chunk_begin.cpu().tolist(),
        groups=[tuple(g) for g in bufs.groups[:ng].cpu().tolist()],
        group_begin=bufs.group_begin.cpu().tolist(),
        device_rows=bufs.device_rows.cpu().tolist(),
        transfers=[tuple(x) for x in bufs.xfers[:nx].cpu().tolist()],
    )
    return tables, info, (params, bufs, ids_t)


def assert_plan_equal(got: dict, info: dict, ref: "oracle.PlanResult"):
    assert got["loads"] == ref.loads
    assert got["chunks"] == [tuple(c) for c in ref.chunks]
    assert got["chunk_row"] == ref.chunk_row
    assert got["expert_chunk_begin"] == ref.expert_chunk_begin
    assert got["groups"] == [tuple(g) for g in ref.groups]
    assert got["group_begin"] == ref.group_begin
    assert got["device_rows"] == ref.device_rows
    assert got["transfers"] == [tuple(t) for t in ref.transfers]
    assert info["status"] == ref.status
    assert info["n_chunks"] == len(ref.chunks)
    assert info["n_groups"] == len(ref.groups)
    assert info["n_xfers"] == len(ref.transfers)
    assert info["forced"] == ref.forced
    assert info["bypassed"] == int(ref.bypassed)
    assert info["max_device"] == ref.max_device
    assert info["total_rows"] == sum(ref.device_rows)


def rel_err(got: np.ndarray, want: np.ndarray) -> float:
    """max |got - want| / max |want| (over the compared entries)."""
    den = np.abs(want).max()
    return float(np.abs(got.astype(np.float64) - want).max() / (den if den > 0 else 1.0))


def elementwise_rel_err(got: np.ndarray, want: np.ndarray) -> float:
    """Diagnostic, not a bound: max over entries of |got - want| / max(|want|,
    1e-3 max |want|), the per-element relative error with entries near zero
    measured against a floor of a thousandth of the largest one."""
    want = np.asarray(want, dtype=np.float64)
    den = np.maximum(np.abs(want), 1e-3 * max(np.abs(want).max(), 1e-300))
    return float((np.abs(got.astype(np.float64) - want) / den).max())


def report(tag: str, got: np.ndarray, want: np.ndarray) -> float:
    """Print the bound's relative error and the element-wise diagnostic;
    returns the former."""
    err = rel_err(got, want)
    print(f"[{tag}] max-norm rel err {err:.3e}, element-wise rel err "
          f"{elementwise_rel_err(got, want):.3e}", flush=True)
    return err


class LayerRun:
    """Inputs on the GPU, packed weights, and one LLEPLayer."""

    def __init__(self, cfg, seed=0, dev="cuda:0", mode="llep", weights=True):
        import torch
        from paper_2601_17111_amd import binding as B
        from paper_2601_17111_amd.layer import LLEPLayer
        from paper_2601_17111_amd.synth import make_inputs, make_weights
        self.cfg, self.seed, self.dev = cfg, seed, dev
        self.inp = make_inputs(cfg, seed)
        self.tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
        self.ids = torch.from_numpy(self.inp.ids).to(dev)
        self.gates = torch.from_numpy(self.inp.gates).to(dev)
        self.x = torch.from_numpy(self.inp.x).to(dev).to(self.tdt)
        self.layer = LLEPLayer(cfg.T, cfg.K, cfg.E, cfg.P, cfg.D, cfg.F, cfg.capacity,
                               self.tdt, dev, cfg.min_chunk, cfg.lam, mode)
        if weights:
            self.wg, self.wu, self.wd = make_weights(cfg, seed, device=dev)
            self.gu, self.dn = B.llep_pack_weights(self.wg, self.wu, self.wd)
            torch.cuda.synchronize()

    def host_weights(self, experts):
        """float32 host copies of the given experts' weights."""
        return {int(e): (self.wg[e].float().cpu().numpy(), self.wu[e].float().cpu().numpy(),
                         self.wd[e].float().cpu().numpy()) for e in experts}

    def forward(self, device=-1):
        import torch
        from paper_2601_17111_amd import binding as B
        self.layer.forward(self.ids, self.gates, self.x, self.gu, self.dn, device)
        torch.cuda.synchronize()
        # no down-projection tile gave up waiting for its activations
        assert not self.layer.bufs.info_dict()["status"] & B.LLEP_STATUS_FFN_WAIT
        return self.layer.y
