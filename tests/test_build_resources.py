"""Compiler resource checks on the gfx950 code objects (CPU only: hipcc
cross-compiles). Every kernel must build without scratch memory or VGPR
spills, and fit the 160 KiB of LDS of a compute unit; and no inline asm may
rely on a clobber of a register the compiler reserves (m0: such a clobber is
not honoured, so a value the compiler keeps there would be overwritten)."""

import os
import re
import shutil
import subprocess

import pytest

from paper_2601_17111_amd import _build

HIP_SOURCES = [s for s in _build.SOURCES if s.endswith(".hip")]


def _resources(src, tmp_path):
    if not os.path.exists(_build.HIPCC) and shutil.which("hipcc") is None:
        pytest.skip("hipcc not available")
    out = tmp_path / (os.path.splitext(src)[0] + ".dev.o")
    cmd = [_build.HIPCC, *_build.FLAGS, "--cuda-device-only", "-c",
           os.path.join(_build.CSRC, src), "-o", str(out),
           "-Rpass-analysis=kernel-resource-usage"]
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert p.returncode == 0, p.stdout
    assert "clobber list contains reserved registers" not in p.stdout, p.stdout
    kernels, cur = {}, None
    for line in p.stdout.splitlines():
        m = re.search(r"remark:\s+Function Name: (\S+)", line)
        if m:
            cur = kernels.setdefault(m.group(1), {})
            continue
        m = re.search(r"remark:\s+([A-Za-z ]+?)(?: \[[^\]]*\])?: (\w+) \[-Rpass", line)
        if m and cur is not None:
            cur[m.group(1).strip()] = m.group(2)
    return kernels


@pytest.mark.parametrize("src", HIP_SOURCES)
def test_no_scratch_no_vgpr_spills(src, tmp_path):
    kernels = _resources(src, tmp_path)
    assert kernels, "no kernel resource remarks parsed"
    for name, r in kernels.items():
        assert r.get("ScratchSize") == "0", (name, r)
        assert r.get("VGPRs Spill") == "0", (name, r)
        assert int(r.get("LDS Size", "0")) <= 160 * 1024, (name, r)
