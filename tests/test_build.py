"""Build-level guard (CPU): the step kernels compile for gfx950 without
register spills.  A spill puts per-lane scratch traffic into the streaming
loop, which costs bandwidth the step cannot spare."""
import os
import re
import shutil
import subprocess

import pytest

from paper_2508_01744_amd import _build

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not shutil.which(HIPCC) and not os.path.exists(HIPCC), reason="hipcc not found")
def test_step_kernels_do_not_spill(tmp_path):
    src = os.path.join(_build.CSRC, "agft_step.hip")
    flags = [f for f in _build.HIPCC_FLAGS if f != "-shared"]
    cmd = [HIPCC, *flags, "-c", "-I", _build.INCLUDE, src, "-o", str(tmp_path / "step.o"),
           "-Rpass-analysis=kernel-resource-usage"]
    out = subprocess.run(cmd, capture_output=True, text=True, check=True).stderr
    kernels = re.findall(r"Function Name: (\S*agft_step_kernel\S*)(.*?)(?=Function Name:|\Z)", out, re.S)
    # d = 8, 16, 32, each with packed and padded tails; d = 16 packed also at
    # six wavefronts per SIMD; each for one- and four-wavefront workgroups,
    # with and without the simulator's environment in the epilogue
    assert len(kernels) == 28, out[-2000:]
    for name, body in kernels:
        scratch = int(re.search(r"ScratchSize \[bytes/lane\]: (\d+)", body).group(1))
        assert scratch == 0, f"{name} spills {scratch} bytes per lane"
