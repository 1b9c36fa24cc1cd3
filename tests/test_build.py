"""Build-level guards (CPU): the step kernels compile for gfx950 without
register spills (a spill puts per-lane scratch traffic into the streaming
loop, which costs bandwidth the step cannot spare), and the bench's
stream-ceiling library is built and checks its arguments."""
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


def test_stream_ceiling_library_checks_its_arguments():
    """The bench's ceiling library is built beside the tuner's, exports its
    two entry points and rejects out-of-range arguments before any HIP call."""
    import ctypes
    assert os.path.exists(_build.CEILING_LIB), "run __graft_entry__.build()"
    lib = ctypes.CDLL(_build.CEILING_LIB)
    dp = ctypes.POINTER(ctypes.c_double)
    f = lib.agft_stream_ceiling
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, dp, dp]
    g = lib.agft_stream_ceiling_at
    g.restype = ctypes.c_int
    g.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, dp, dp]
    a, b = ctypes.c_double(), ctypes.c_double()
    for args in ((0, 4864, 38, 1), (1 << 31, 4864, 38, 1), (1, 0, 1, 1), (1, 4864, 0, 1), (1, 4864, 257, 1),
                 (1, 10, 38, 1), (1, 4864, 38, 0)):
        assert f(*args, ctypes.byref(a), ctypes.byref(b)) == 1, args
        assert g(*args, 0, ctypes.byref(a), ctypes.byref(b)) == 1, args
    assert f(1, 4864, 38, 1, None, ctypes.byref(b)) == 1
    assert g(1, 4864, 38, 1, -1, ctypes.byref(a), ctypes.byref(b)) == 1
    assert g(1, 4864, 38, 1, 65, ctypes.byref(a), ctypes.byref(b)) == 1
    assert g(1, 4864, 38, 1, 4, ctypes.byref(a), None) == 1
