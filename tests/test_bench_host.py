"""bench.py's contract on the host: one GPU only (N > 1 exits with a message
and status 2, before touching the GPU), and the flags the driver and the
profiles use are accepted."""

import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True, timeout=120)


def test_more_than_one_gpu_is_refused():
    p = _run("--gpus", "2", "--steps", "1", "--warmup", "0")
    assert p.returncode == 2
    assert "one GPU" in p.stderr
    assert p.stdout.strip() == ""


def test_sweeps_refuse_more_than_one_gpu():
    for sweep in ("alpha", "experts"):
        p = _run("--gpus", "8", "--sweep", sweep)
        assert p.returncode == 2


def test_flags_parse():
    sys.path.insert(0, ROOT)
    import bench
    old = sys.argv
    try:
        sys.argv = ["bench.py", "--steps", "3", "--warmup", "1", "--no-ep", "--no-cpu-baseline",
                    "--no-backward", "--no-full-layer", "--copy-calibration", "--workload",
                    "deepseek-v3"]
        a = bench._parse()
    finally:
        sys.argv = old
    assert (a.steps, a.warmup, a.no_ep, a.no_backward, a.no_full_layer) == (3, 1, True, True, True)
    assert bench._config(a.workload).E == 256
    # the committed traffic figure belongs to the default workload only
    assert bench._traffic("deepseek-v3") is None


def test_kernel_hash_ignores_comments_only():
    """The traffic figure is keyed by a hash of the GEMM source that ignores
    comments and spacing but not code."""
    sys.path.insert(0, ROOT)
    import bench
    a = bench._code_only('int x = 1;  // one\n/* two\n three */ int y = "//" [0];\n')
    b = bench._code_only('int x = 1;\n\n   int y = "//" [0]; // other words\n')
    c = bench._code_only('int x = 2;\nint y = "//" [0];\n')
    assert a == b
    assert a != c
    assert '"//"' in a
