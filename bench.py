"""Benchmark of the LLEP expert-layer hot path on one MI355X.

A step is one pass of the whole path over one batch of synthetic input, all
on one stream: plan (histogram + least-loaded assignment) -> permute ->
grouped SwiGLU FFN of the most-loaded virtual device's groups -> combine.
Inputs are resident in HBM before timing starts; the most-loaded device d* is
read from the plan once, before timing (the batch does not change).

Timing: every timed step follows a 512 MiB cache-flush write (outside the
step's events, so no step finds the previous one's operands in the L2s or the
256 MB MALL); the reported times are medians over the timed steps of HIP
events on the stream, with their spread.

Prints one JSON line. `value` is tokens per second of the measured step
(T / median time per step). The `roofline` object is for the grouped FFN
(a tiny tile-list kernel, then one persistent launch for both projections):
algorithmic flops 6*D*F per row of d*, over the median duration of that call
measured with HIP events on its stream. `cpu_baseline` times the CPU oracle on
a bounded sample of the same workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "MoE-layer tokens/s + grouped-GEMM % bf16 MFMA peak, max-loaded share, 1 GPU"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA (vendor figure)
PEAK_HBM_GBPS = 8000.0      # MI355X HBM3E (vendor figure)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "grouped_ffn_traffic.json")


def _parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="gpt-oss-120b-hot1")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-sample-rows", type=int, default=65536,
                    help="cap on the rows of the most-loaded device the CPU oracle computes "
                         "(all of them when fewer; the time is scaled to all rows otherwise)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ep", action="store_true", help="skip the standard-EP comparison")
    ap.add_argument("--no-backward", action="store_true", help="skip the backward measurement")
    ap.add_argument("--no-full-layer", action="store_true",
                    help="skip the all-devices grouped FFN measurement")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="before warmup, run a plain 1 GiB -> 1 GiB elementwise copy (torch.neg on "
                         "float32) three times: a kernel of known traffic that scales the HBM "
                         "counters of a rocprofv3 --pmc run of this command")
    ap.add_argument("--sweep", choices=["alpha", "lambda", "batch", "all", "experts"],
                    help="instead of the bench line: the planner-knob and batch sweeps of the "
                         "paper's ablations on the gpt-oss-120b layer shape, one JSON line per "
                         "point (LLEP vs standard EP, P-device model)")
    return ap.parse_args()


def _config(name):
    from paper_2601_17111_amd.synth import CONFIGS, gpt_oss_120b
    if name.startswith("gpt-oss-120b-hot"):
        return gpt_oss_120b(int(name[len("gpt-oss-120b-hot"):]))
    return CONFIGS[name]


def _code_only(text: str) -> str:
    """C++ source without comments and blank space, so that the hash below
    changes with the code only (string literals are kept as they are)."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c == '"':
            j = i + 1
            while j < n and text[j] != '"':
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            while i < n and text[i] != "\n":
                i += 1
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def _kernel_hash():
    """Hash of the grouped-FFN kernel source (comments and spacing ignored):
    the traffic figure is used only while the code it was measured on is
    unchanged."""
    h = hashlib.sha256()
    for f in ("gemm.h", "grouped_ffn.hip", "common.h"):
        with open(os.path.join(ROOT, "paper_2601_17111_amd", "csrc", f), encoding="utf-8") as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def _traffic(workload):
    """Measured HBM bytes per grouped-FFN call from the committed counter
    summary, if it was taken on this workload with the current kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_hash") != _kernel_hash() or t.get("workload") != workload:
        return None
    return t.get("bytes_per_call")


def _m_local_gb(layer, P, D, F, eb):
    """Peak memory model of each device's share (Sec. 3.2, Eq. 4, with the
    SwiGLU expert's three weight matrices) from the plan's group table, GB."""
    from paper_2601_17111_amd.layer import m_local_bytes
    info = layer.bufs.info_dict()
    groups = layer.bufs.groups[:info["n_groups"]].cpu().tolist()
    return [v / 1e9 for v in m_local_bytes(groups, P, D, F, eb)]


FLUSH_BYTES = 512 << 20  # written between timed reps: twice the 256 MB MALL


class _Flush:
    """A device buffer of FLUSH_BYTES, overwritten before each timed rep so
    that no rep finds its operands in the L2s or the MALL from the previous
    one (the write is outside the timed events)."""

    def __init__(self, dev):
        import torch
        self.buf = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device=dev)
        self.i = 0

    def __call__(self):
        self.i += 1
        self.buf.fill_(self.i & 0xFF)


def _stats(vals):
    """Median and spread of a list of per-rep times (ms)."""
    v = sorted(vals)
    n = len(v)

    def q(f):
        return v[min(n - 1, int(round(f * (n - 1))))]
    return {"median": q(0.5), "mean": sum(v) / n, "min": v[0], "p10": q(0.1), "p90": q(0.9),
            "max": v[-1], "reps": n}


def _time_steps(layer, run, steps, dstar, flush=None, spread=None):
    """Run `steps` steps, each after a cache-flush write (outside its
    events); per-segment HIP event times (ms) on the stream. Returns the
    median step time and the per-segment medians; `spread`, if a dict, gets
    the statistics of the step and segment times."""
    import torch
    names = ("plan", "permute", "grouped_ffn", "combine")
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(steps)]
    torch.cuda.synchronize()
    for i in range(steps):
        if flush is not None:
            flush()
        e = ev[i]
        e[0].record()
        layer.plan(run["ids"])
        e[1].record()
        layer.permute(run["ids"], run["gates"], run["x"])
        e[2].record()
        layer.ffn(run["gu"], run["dn"], dstar)
        e[3].record()
        layer.combine(run["gates"])
        e[4].record()
    torch.cuda.synchronize()
    per = {k: [e[j].elapsed_time(e[j + 1]) for e in ev] for j, k in enumerate(names)}
    tot = [e[0].elapsed_time(e[4]) for e in ev]
    if spread is not None:
        spread["step"] = _stats(tot)
        for k in names:
            spread[k] = _stats(per[k])
    return _stats(tot)["median"], {k: _stats(per[k])["median"] for k in names}


def _backward(layer, run, wg, wu, wd, cfg, dstar, n_rows, steps, flush):
    """The backward of the step on the most-loaded device's share: combine
    backward (all tokens) -> grouped SwiGLU backward of d*'s groups (input
    gradients of its rows and its partial weight gradients) from the gate /
    up values the training forward kept -> the pairs' input gradients summed
    per token. Also timed: the same backward recomputing gate / up, and the
    training forward's grouped FFN on d* (which keeps them). HIP event times
    per segment (ms)."""
    import torch
    from paper_2601_17111_amd import binding as B
    gut, dnt = B.llep_pack_weights_backward(wg, wu, wd)
    g = torch.Generator(device=run["x"].device)
    g.manual_seed(7)
    dy = torch.randn(cfg.T, cfg.D, generator=g, device=run["x"].device).to(torch.bfloat16)
    layer.forward(run["ids"], run["gates"], run["x"], run["gu"], run["dn"], -1,
                  save_gate_up=True)
    layer.backward(dy, run["gates"], run["gu"], gut, dnt, dstar)  # allocates the buffers
    L = layer

    def step(gate_up, e):
        """One backward step; e[0..3] are recorded around its three calls."""
        e[0].record()
        B.llep_combine_backward(L.params, L.out_perm, L.pair_row, run["gates"], dy, L.d_out_perm,
                                L.d_gates)
        e[1].record()
        B.llep_grouped_ffn_backward(L.params, L.bufs, dstar, L.x_perm, L.d_out_perm, run["gu"],
                                    gut, dnt, L.dx_perm, L.dw_gate, L.dw_up, L.dw_down,
                                    L.bwd_workspace, gate_up=gate_up)
        e[2].record()
        B.llep_combine(L.params, L.dx_perm, L.pair_row, None, L.dx)
        e[3].record()

    def timed(gate_up):
        names = ("combine_backward", "grouped_ffn_backward", "dx_sum")
        per = {k: [] for k in names}
        for i in range(steps + 2):
            flush()
            e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
            step(gate_up, e)
            torch.cuda.synchronize()
            if i >= 2:
                for k, (a, b) in zip(names, zip(e[:-1], e[1:])):
                    per[k].append(a.elapsed_time(b))
        return {k: _stats(v)["median"] for k, v in per.items()}

    seg = timed(L.gate_up)
    recompute_ms = timed(None)["grouped_ffn_backward"]
    # the training forward's grouped FFN on d*: the inference one plus the
    # stores of gate / up
    train = []
    for i in range(steps + 2):
        flush()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        L.ffn(run["gu"], run["dn"], dstar, save_gate_up=True)
        b.record()
        torch.cuda.synchronize()
        if i >= 2:
            train.append(a.elapsed_time(b))
    train_ms = _stats(train)["median"]
    D, F, T, K = cfg.D, cfg.F, cfg.T, cfg.K
    R = T * K
    t_ffn = seg["grouped_ffn_backward"] * 1e-3
    cb_bytes = T * D * 2 + 2 * R * D * 2 + 12 * R
    # every expert with rows on d* gets its full float32 weight gradients
    # (3 D F values), however few its rows: bytes the flop count leaves out
    gb = L.bufs.group_begin.cpu().tolist()
    experts = {int(e) for e in L.bufs.groups[gb[dstar]:gb[dstar + 1], 1].cpu().tolist()}
    wgrad_bytes = len(experts) * 3 * D * F * 4
    floor_s = 12.0 * D * F * n_rows / (PEAK_BF16_TFLOPS * 1e12) + wgrad_bytes / (PEAK_HBM_GBPS * 1e9)
    del gut, dnt
    L.gate_up = None
    return {
        "ms_per_step": sum(seg.values()), "segments_ms": seg, "device": dstar, "rows": n_rows,
        # 12 D F per row: the backward of the three projections (twice the
        # forward); recomputing gate / up adds 4 D F
        "grouped_ffn_backward_TFLOPs": 12.0 * D * F * n_rows / t_ffn / 1e12,
        "grouped_ffn_backward_frac": 12.0 * D * F * n_rows / t_ffn / 1e12 / PEAK_BF16_TFLOPS,
        # the MFMA work at the bf16 peak plus the float32 weight-gradient
        # writes at the HBM peak, one after the other, over the measured time
        "grouped_ffn_backward_experts": len(experts),
        "grouped_ffn_backward_weight_gradient_GB": wgrad_bytes / 1e9,
        "grouped_ffn_backward_floor_ms": floor_s * 1e3,
        "grouped_ffn_backward_floor_frac": floor_s / t_ffn,
        "grouped_ffn_backward_recompute_ms": recompute_ms,
        "grouped_ffn_backward_recompute_TFLOPs":
            16.0 * D * F * n_rows / (recompute_ms * 1e-3) / 1e12,
        "grouped_ffn_train_forward_ms": train_ms,
        "combine_backward_GBps": cb_bytes / (seg["combine_backward"] * 1e-3) / 1e9,
        "tokens_per_s": T / (sum(seg.values()) * 1e-3),
    }


def _cpu_baseline(cfg, inp, expert_weights, args):
    """The oracle on the host over the whole step: plan and permutation over
    all pairs (Python, one core), the SwiGLU expert function (float64 numpy
    BLAS) over every row of the most-loaded device (a sample scaled to all of
    them only past --cpu-sample-rows), and the gate-weighted sum over every
    token (in chunks of 4096 tokens, inputs drawn outside the timed part)."""
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        blas = 1
    flat = inp.ids.reshape(-1).tolist()
    t0 = time.perf_counter()
    pl = oracle.plan(flat, cfg.E, cfg.P, cfg.capacity, cfg.min_chunk, lam=cfg.lam)
    t_plan = time.perf_counter() - t0
    t0 = time.perf_counter()
    _, row_pair = oracle.permute(flat, pl, cfg.E)
    t_perm = time.perf_counter() - t0
    dstar = pl.max_device
    groups = pl.groups[pl.group_begin[dstar]:pl.group_begin[dstar + 1]]
    n_rows = pl.device_rows[dstar]
    # sample rows of d*, spread over its groups in proportion to their size
    rng = np.random.default_rng(0)
    row0 = groups[0][2] if groups else 0
    rows = row0 + np.sort(rng.choice(n_rows, size=min(args.cpu_sample_rows, n_rows), replace=False))
    weights = {int(e): expert_weights(int(e)) for (_, e, _, _) in groups}
    t0 = time.perf_counter()
    for (d, e, r0, n) in groups:
        sel = rows[(rows >= r0) & (rows < r0 + n)]
        if len(sel) == 0:
            continue
        xs = inp.x[row_pair[sel] // cfg.K]
        oracle.swiglu_ffn(xs, *weights[int(e)])
    t_ffn = (time.perf_counter() - t0) * n_rows / max(1, len(rows))
    t_comb = 0.0
    for t_lo in range(0, cfg.T, 4096):
        t_hi = min(cfg.T, t_lo + 4096)
        pair_out = rng.standard_normal((t_hi - t_lo, cfg.K, cfg.D))
        t0 = time.perf_counter()
        oracle.combine(pair_out, inp.gates[t_lo:t_hi])
        t_comb += time.perf_counter() - t0
    total = t_plan + t_perm + t_ffn + t_comb
    return {
        "value": cfg.T / total, "unit": "tokens/s", "cores": int(max(1, blas)),
        "kind": "oracle",
        "sample": (f"plan + permutation over all {cfg.R} pairs (Python, 1 core); "
                   f"float64 SwiGLU over {len(rows)} of the {n_rows} rows of the most-loaded "
                   f"device" + (", scaled to all of them" if len(rows) < n_rows else "") +
                   f" (numpy BLAS, {blas} threads); gate-weighted sum over all {cfg.T} tokens"),
        "seconds": {"plan": t_plan, "permute": t_perm, "ffn": t_ffn, "combine": t_comb},
        "host_cores": len(os.sched_getaffinity(0)),
    }


def _sweep(args):
    """Ablation sweeps (Sec. 5.3 factor alpha, adaptive ratio lambda, batch size)
    on the gpt-oss-120b layer shape with a hot set of 4 experts: per point the
    most-loaded device's rows and the P-device model time of LLEP and of
    standard EP. Communication is not modelled (one GPU)."""
    import torch
    from fractions import Fraction
    from paper_2601_17111_amd import binding as B
    from paper_2601_17111_amd.layer import LLEPLayer
    from paper_2601_17111_amd.synth import CONFIGS, make_inputs, make_weights

    B.lib()
    dev = "cuda:0"
    base = CONFIGS["gpt-oss-120b"].with_(lam=1.3, min_chunk=1024, alpha=Fraction(1))
    wg, wu, wd = make_weights(base, args.seed, device=dev)
    gu, dn = B.llep_pack_weights(wg, wu, wd)
    del wg, wu, wd
    points = []
    if args.sweep in ("alpha", "all"):
        for frac in (0.3, 0.5, 0.8, 0.95):
            for a in ("1", "3/2", "2", "5/2", "3"):
                points.append(("alpha", base.with_(routing=("hot", frac, 4), alpha=Fraction(a))))
    if args.sweep in ("lambda", "all"):
        for frac in (0.15, 0.2, 0.3, 0.5):
            for lam in (1.1, 1.4, 1.7, 2.0, 2.3, 2.6):
                points.append(("lambda", base.with_(T=8192, routing=("hot", frac, 4), lam=lam)))
    if args.sweep in ("batch", "all"):
        for frac in (0.3, 0.5, 0.8, 0.95):
            for T in (4096, 8192, 16384, 32768, 65536):
                points.append(("batch", base.with_(T=T, routing=("hot", frac, 4))))
    steps = max(5, args.steps // 4)
    flush = _Flush(dev)
    for kind, cfg in points:
        inp = make_inputs(cfg, args.seed)
        run = dict(ids=torch.from_numpy(inp.ids).to(dev), gates=torch.from_numpy(inp.gates).to(dev),
                   x=torch.from_numpy(inp.x).to(dev).to(torch.bfloat16), gu=gu, dn=dn)
        res = {}
        for mode in ("llep", "ep"):
            layer = LLEPLayer(cfg.T, cfg.K, cfg.E, cfg.P, cfg.D, cfg.F, cfg.capacity, torch.bfloat16,
                              dev, cfg.min_chunk, cfg.lam, mode)
            layer.plan(run["ids"])
            torch.cuda.synchronize()
            info = layer.bufs.info_dict()
            d = info["max_device"]
            rows = layer.bufs.device_rows.cpu().tolist()[d]
            for _ in range(2):
                layer.plan(run["ids"]); layer.permute(run["ids"], run["gates"], run["x"])
                layer.ffn(gu, dn, d); layer.combine(run["gates"])
            _, seg = _time_steps(layer, run, steps, d, flush)
            model = seg["plan"] + (seg["permute"] + seg["combine"]) / cfg.P + seg["grouped_ffn"]
            res[mode] = {"max_device_rows": rows, "bypassed": info["bypassed"],
                         "forced": info["forced"], "n_xfers": info["n_xfers"],
                         "segments_ms": seg, "model_ms": model}
            del layer
        print(json.dumps({
            "sweep": kind, "T": cfg.T, "hot_frac": cfg.routing[1], "hot_experts": cfg.routing[2],
            "alpha": str(cfg.alpha), "lambda": cfg.lam, "min_chunk": cfg.min_chunk,
            "capacity": cfg.capacity, "llep": res["llep"], "ep": res["ep"],
            "speedup_model": res["ep"]["model_ms"] / res["llep"]["model_ms"],
            "speedup_ffn": res["ep"]["segments_ms"]["grouped_ffn"] /
                           res["llep"]["segments_ms"]["grouped_ffn"],
        }), flush=True)


def _sweep_experts(args):
    """App. A.1: the same work split evenly over N experts. 65536 tokens, one
    expert each, D = F = 8192, all experts on one device (P = 1), N in
    4 .. 256; the grouped SwiGLU FFN over all rows, timed with HIP events.
    Weights are drawn and packed 16 experts at a time."""
    import torch
    from fractions import Fraction
    from paper_2601_17111_amd import binding as B
    from paper_2601_17111_amd.layer import LLEPLayer
    from paper_2601_17111_amd.synth import LayerConfig, make_inputs, make_weights

    B.lib()
    dev = "cuda:0"
    T, D, F = 65536, 8192, 8192
    reps = max(5, args.steps // 4)
    flush = _Flush(dev)
    for N in (4, 16, 32, 64, 128, 256):
        cfg = LayerConfig(f"a1-n{N}", T=T, D=D, F=F, E=N, K=1, P=1, alpha=Fraction(1),
                          dtype="bf16", routing=("balanced",))
        gu = torch.empty((N, 2 * F, D), dtype=torch.bfloat16, device=dev)
        dn = torch.empty((N, D, F), dtype=torch.bfloat16, device=dev)
        for b0 in range(0, N, 16):
            nb = min(16, N - b0)
            wg, wu, wd = make_weights(cfg.with_(E=nb), args.seed + b0, device=dev)
            B.llep_pack_weights(wg, wu, wd, out=(gu[b0:b0 + nb], dn[b0:b0 + nb]))
            del wg, wu, wd
        inp = make_inputs(cfg, args.seed)
        ids = torch.from_numpy(inp.ids).to(dev)
        gates = torch.from_numpy(inp.gates).to(dev)
        x = torch.from_numpy(inp.x).to(dev).to(torch.bfloat16)
        layer = LLEPLayer(T, 1, N, 1, D, F, cfg.capacity, torch.bfloat16, dev)
        layer.plan(ids)
        layer.permute(ids, gates, x)
        for _ in range(2):
            layer.ffn(gu, dn, -1)
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            flush()
            s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s.record()
            layer.ffn(gu, dn, -1)
            e.record()
            torch.cuda.synchronize()
            ts.append(s.elapsed_time(e))
        ms = sorted(ts)[len(ts) // 2]
        flops = 6.0 * D * F * T
        print(json.dumps({"sweep": "experts", "experts": N, "tokens": T, "D": D, "F": F,
                          "rows_per_expert": T // N, "grouped_ffn_ms": ms,
                          "TFLOPs": flops / (ms * 1e-3) / 1e12,
                          "frac_of_peak": flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS}),
              flush=True)
        del gu, dn, layer
        torch.cuda.empty_cache()


def main():
    args = _parse()
    if args.sweep == "experts":
        if args.gpus != 1:
            print("the sweeps run on one GPU", file=sys.stderr)
            sys.exit(2)
        _sweep_experts(args)
        return
    if args.sweep:
        if args.gpus != 1:
            print("the sweeps run on one GPU", file=sys.stderr)
            sys.exit(2)
        _sweep(args)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the P devices of the "
              f"plan are virtual devices on that GPU.", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2601_17111_amd import binding as B
    from paper_2601_17111_amd.layer import LLEPLayer
    from paper_2601_17111_amd.synth import make_inputs, make_weights

    B.lib()
    dev = "cuda:0"
    cfg = _config(args.workload)
    inp = make_inputs(cfg, args.seed)
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    run = dict(ids=torch.from_numpy(inp.ids).to(dev), gates=torch.from_numpy(inp.gates).to(dev),
               x=torch.from_numpy(inp.x).to(dev).to(tdt))
    wg, wu, wd = make_weights(cfg, args.seed, device=dev)
    run["gu"], run["dn"] = B.llep_pack_weights(wg, wu, wd)
    layer = LLEPLayer(cfg.T, cfg.K, cfg.E, cfg.P, cfg.D, cfg.F, cfg.capacity, tdt, dev,
                      cfg.min_chunk, cfg.lam, "llep")

    def plan_info():
        layer.plan(run["ids"])
        torch.cuda.synchronize()
        info = layer.bufs.info_dict()
        rows = layer.bufs.device_rows.cpu().tolist()
        return info, rows

    # untimed: the plan's most-loaded device and its groups
    info, dev_rows = plan_info()
    dstar = info["max_device"]
    layer.permute(run["ids"], run["gates"], run["x"])
    torch.cuda.synchronize()
    n_rows = dev_rows[dstar]

    if args.copy_calibration:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    flush = _Flush(dev)
    for _ in range(args.warmup):
        flush()
        layer.plan(run["ids"])
        layer.permute(run["ids"], run["gates"], run["x"])
        layer.ffn(run["gu"], run["dn"], dstar)
        layer.combine(run["gates"])
    spread = {}
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    ms, seg = _time_steps(layer, run, args.steps, dstar, flush, spread)
    t_wall = time.perf_counter() - t_wall

    D, F, T, K = cfg.D, cfg.F, cfg.T, cfg.K
    eb = 2 if cfg.dtype == "bf16" else 4
    flops = 6.0 * D * F * n_rows
    tflops = flops / (seg["grouped_ffn"] * 1e-3) / 1e12
    R = T * K
    perm_bytes = T * D * eb + R * D * eb + 12 * R
    comb_bytes = R * D * eb + T * D * eb + 8 * R
    traffic = _traffic(args.workload)
    out = {
        "metric": METRIC,
        "value": T / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {
            "workload": (f"{cfg.name}: MoE layer T={T} D={D} SwiGLU F={F} E={cfg.E} top-{K}, "
                         f"P={cfg.P} virtual devices, capacity {cfg.capacity} "
                         f"(alpha={cfg.alpha}), routing {cfg.routing}, seed {args.seed}; "
                         f"step = plan + permute + grouped FFN of device {dstar} + combine"),
            "global_batch": T, "parallelism": "1 GPU, P virtual devices",
        },
        "roofline": {
            "bound": "mfma", "achieved": tflops, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": tflops / PEAK_BF16_TFLOPS, "traffic": traffic,
            "kernel": ("llep_grouped_ffn on the most-loaded device (tile_table_kernel + "
                       "ffn_fused_kernel: both projections in one persistent launch)"),
            "flops_per_launch": flops,
        },
        "segments_ms": seg,
        "timing": {"statistic": "median over the timed steps of HIP-event times on the stream",
                   "flush_bytes_between_steps": FLUSH_BYTES, "spread_ms": spread,
                   "wall_s_incl_flushes": t_wall},
        "plan": {"max_device": dstar, "device_rows": dev_rows, "capacity": cfg.capacity,
                 "n_chunks": info["n_chunks"], "n_groups": info["n_groups"],
                 "n_xfers": info["n_xfers"]},
        "permute_GBps": perm_bytes / (seg["permute"] * 1e-3) / 1e9,
        "combine_GBps": comb_bytes / (seg["combine"] * 1e-3) / 1e9,
    }
    out["permute_hbm_frac"] = out["permute_GBps"] / PEAK_HBM_GBPS
    out["combine_hbm_frac"] = out["combine_GBps"] / PEAK_HBM_GBPS
    # P-device model of the layer: permute/combine are split evenly over the
    # P source devices, the expert GEMMs wait for the most-loaded device
    model_ms = seg["plan"] + (seg["permute"] + seg["combine"]) / cfg.P + seg["grouped_ffn"]
    out["layer_tokens_per_s_p_device_model"] = T / (model_ms * 1e-3)

    m_llep = _m_local_gb(layer, cfg.P, D, F, eb)
    out["m_local_GB"] = {"llep_max": max(m_llep), "llep_per_device": m_llep}

    # the raw 1-GPU layer: all P devices' groups back to back in one call
    if not args.no_full_layer:
        ms_full, seg_full = _time_steps(layer, run, max(5, args.steps // 3), -1, flush)
        total_rows = sum(dev_rows)
        out["full_layer_all_devices"] = {
            "ms_per_step": ms_full, "tokens_per_s": T / (ms_full * 1e-3), "segments_ms": seg_full,
            "rows": total_rows,
            "grouped_ffn_TFLOPs": 6.0 * D * F * total_rows / (seg_full["grouped_ffn"] * 1e-3) / 1e12,
        }

    if cfg.dtype == "bf16" and not args.no_backward:
        out["backward"] = _backward(layer, run, wg, wu, wd, cfg, dstar, n_rows,
                                    max(5, args.steps // 2), flush)

    if not args.no_ep:
        layer.set_mode("ep")
        info_ep, rows_ep = plan_info()
        d_ep = info_ep["max_device"]
        m_ep = _m_local_gb(layer, cfg.P, D, F, eb)
        out["m_local_GB"].update({"ep_max": max(m_ep), "ep_per_device": m_ep,
                                  "ep_over_llep": max(m_ep) / max(m_llep)})
        layer.permute(run["ids"], run["gates"], run["x"])
        for _ in range(2):
            layer.ffn(run["gu"], run["dn"], d_ep)
        ms_ep, seg_ep = _time_steps(layer, run, max(5, args.steps // 3), d_ep, flush)
        out["standard_ep"] = {
            "max_device": d_ep, "max_device_rows": rows_ep[d_ep], "ms_per_step": ms_ep,
            "segments_ms": seg_ep,
            "grouped_ffn_TFLOPs": 6.0 * D * F * rows_ep[d_ep] / (seg_ep["grouped_ffn"] * 1e-3) / 1e12,
        }
        out["speedup_llep_vs_ep"] = {
            "step": ms_ep / ms, "grouped_ffn": seg_ep["grouped_ffn"] / seg["grouped_ffn"]}
        layer.set_mode("llep")

    if not args.no_cpu_baseline:
        def expert_weights(e):
            return (wg[e].float().cpu().numpy(), wu[e].float().cpu().numpy(),
                    wd[e].float().cpu().numpy())
        out["cpu_baseline"] = _cpu_baseline(cfg, inp, expert_weights, args)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
