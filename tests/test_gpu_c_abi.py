"""The C ABI from a plain C caller (tests/c_abi/agft_c_example.c): it owns
its device buffers, runs a tuner with contexts and rewards of its own and
records them; the same inputs replayed through the Python binding give the
same actions, and the oracle agrees with both."""
import os
import subprocess

import numpy as np
import pytest

import parity
from gpu_helpers import run_open_loop, say

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "agft_c_example")


@pytest.mark.parametrize("B,K,d,T", [(8, 24, 8, 60), (5, 40, 16, 50), (3, 33, 32, 40)])
def test_c_caller(B, K, d, T, tmp_path):
    assert os.path.exists(EXE), f"{EXE} is missing: build() compiles it"
    rec = tmp_path / "run.bin"
    say(f"[c-abi] B={B} K={K} d={d} T={T}")
    res = subprocess.run([EXE, str(B), str(K), str(d), str(T), str(rec)], capture_output=True,
                         text=True, timeout=120)
    assert res.returncode == 0, res.stderr
    assert f"steps {T} pending 0" in res.stdout, res.stdout
    raw = np.fromfile(rec, dtype=np.int32)
    assert tuple(raw[:4]) == (B, K, d, T)
    per = B * d + B + B
    body = raw[4:].reshape(T, per)
    X = body[:, :B * d].view(np.float32).reshape(T, B, d).astype(np.float64)
    A = body[:, B * d:B * d + B]
    R = body[:, B * d + B:].view(np.float32).astype(np.float64)
    cfg = dict(B=B, K=K, d=d, lam=1.0, alpha0=0.5, sched=0, prune=1, period=10, heuristics=None)
    a, m, s, tuner, _ = run_open_loop(cfg, X, R)
    assert np.array_equal(a, A), "the Python binding decided differently from the C caller"
    st = parity.compare_open_loop("c caller", cfg, X, R, a, m, s)
    say(f"[c-abi] max score err {st['max_score_err']:.2e}, forced {st['forced']}/{st['decisions']}")
