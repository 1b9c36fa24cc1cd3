"""The stream-ceiling library on the GPU: both forms run and time on the cfg4
record layout at a reduced instance count, uncapped and at four workgroups
per compute unit, and the write-back form moves more bytes in no less time
than reading alone."""
import ctypes

import pytest
import torch

from paper_2508_01744_amd import _build

pytestmark = pytest.mark.gpu


def test_stream_ceiling_times_both_forms():
    torch.cuda.init()
    lib = ctypes.CDLL(_build.CEILING_LIB)
    f = lib.agft_stream_ceiling
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                  ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
    r, rw = ctypes.c_double(), ctypes.c_double()
    # 8,192 instances of 128 d = 16 records (4,864 chunks each, 38 per record)
    print("[ceiling] 8192 x 4864 chunks, record 38, 5 launches", flush=True)
    assert f(8192, 4864, 38, 5, ctypes.byref(r), ctypes.byref(rw)) == 0
    print(f"[ceiling] read {r.value:.1f} us, read+writeback {rw.value:.1f} us", flush=True)
    assert 0 < r.value < 1e5 and 0 < rw.value < 1e5
    assert rw.value > 0.9 * r.value


def test_stream_ceiling_at_a_workgroup_cap():
    torch.cuda.init()
    lib = ctypes.CDLL(_build.CEILING_LIB)
    f = lib.agft_stream_ceiling_at
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                  ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
    r, rw = ctypes.c_double(), ctypes.c_double()
    print("[ceiling] 8192 x 4864 chunks, record 38, 5 launches, 4 workgroups per compute unit", flush=True)
    # MI355X: 160 KB of LDS per compute unit admit a 40 KB share per workgroup
    assert f(8192, 4864, 38, 5, 4, ctypes.byref(r), ctypes.byref(rw)) == 0
    print(f"[ceiling] read {r.value:.1f} us, read+writeback {rw.value:.1f} us", flush=True)
    assert 0 < r.value < 1e5 and 0 < rw.value < 1e5
    assert rw.value > 0.9 * r.value
