"""The C ABI library loads, exports every declared symbol and rejects bad
arguments before touching the GPU (CPU only: no call here launches work)."""
import ctypes
import os
import re

import pytest

import paper_2508_01744_amd._lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = []
    for hdr in ("agft.h", "agft_sim.h"):
        text = open(os.path.join(ROOT, "include", hdr)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names += re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\**\s*(agft_[a-z_0-9]+)\s*\(", text, flags=re.M)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    return L.lib()


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(L.EXPORTED)


def test_abi_version_and_strerror(lib):
    assert L.agft_abi_version() == L.ABI_VERSION == 6
    for code in (0, -1, -2, -3, -4):
        assert L.agft_strerror(code)
    assert L.agft_strerror(-99) == "unknown status"


def _cfg(**kw):
    base = dict(B=4, K=16, d=8, lambda_=1.0, alpha0=0.5, alpha_sched=0, prune_rule=0,
                prune_period=50, prune_sticky=1, flags=0)
    base.update(kw)
    return L.agft_config(**base)


def test_state_bytes(lib):
    n = L.agft_state_bytes(_cfg())
    assert n > 0 and n % 256 == 0
    good = dict(prune_rule=15, ext_rounds=60, ext_min_n=3, ext_thr=-1.2, hist_after=30, hist_min_n=6,
                hist_kappa=1.0, hist_min_arms=3, cascade_k=16)
    assert L.agft_state_bytes(_cfg(**good)) == n
    # the arm records dominate: B * K * (d/2) * (d+3)/4 float4 chunks, exactly
    # the d + d(d+1)/2 floats of theta and S per arm, with no padding
    for d, chunks in ((8, 11), (16, 38), (32, 140)):
        assert 4 * chunks == d + d * (d + 1) // 2
        big = L.agft_state_bytes(_cfg(B=4096, K=128, d=d))
        # beyond the records: stats (8 B per arm), instance blocks (<= 256 B),
        # mask words, header and alignment
        assert 0 <= big - 4096 * 128 * chunks * 16 < 4096 * (128 * 8 + 256 + 16) + 1024
    # K is rounded up to whole blocks of 64/d arms: K=125 at d=16 takes 128 slots
    # (the other regions of K=125 add less than the 3 slots' 7.5 MB)
    assert L.agft_state_bytes(_cfg(B=4096, K=125, d=16)) >= 4096 * 128 * 38 * 16
    # with pruning, up to 16 KB of records per exploring instance (26 arms of
    # 608 bytes at d=16) the tails are padded to whole chunks: 40 chunks per
    # record, so K=26 (28 slots of 640 bytes) needs more than K=27 (28 slots
    # of 608)
    b26, b27 = (L.agft_state_bytes(_cfg(B=4096, K=k, d=16, prune_rule=1)) for k in (26, 27))
    assert 4096 * 28 * 40 * 16 <= b26 and b27 < b26 and b27 - 4096 * 28 * 38 * 16 < 4096 * (27 * 8 + 272) + 1024
    # without pruning or refinement every step streams every record: packed
    # tails from 8 KB (14 arms at d=16), so K=26 takes the 608-byte records
    p26 = L.agft_state_bytes(_cfg(B=4096, K=26, d=16))
    assert p26 < b26 and 0 <= p26 - 4096 * 28 * 38 * 16 < 4096 * (26 * 8 + 272) + 1024
    b13, b14 = (L.agft_state_bytes(_cfg(B=4096, K=k, d=16)) for k in (13, 14))
    assert b13 - 4096 * 16 * 40 * 16 >= 0 and b14 < b13
    # the refinement counts the arms in play: K=128 with windows of 21 arms
    # and a coarse grid of 13 streams 12.8 KB, padded tails
    ref = dict(refine=1, refine_period=50, refine_stride=10, refine_half=10, refine_mature=100,
               refine_min_n=4)
    assert L.agft_state_bytes(_cfg(B=4096, K=128, d=16, **ref)) >= 4096 * 128 * 40 * 16
    for bad in (dict(B=0), dict(K=0), dict(K=1025), dict(lambda_=0.0), dict(lambda_=float("nan")),
                dict(alpha0=-1.0), dict(alpha0=float("inf")), dict(alpha_sched=2),
                dict(prune_rule=16), dict(prune_rule=-1), dict(prune_period=0), dict(flags=4), dict(d=12),
                dict(prune_sticky=2), dict(prune_sticky=-1),
                dict(prune_rule=3, prune_sticky=0, ext_rounds=60, ext_min_n=3, ext_thr=-1.2),
                dict(prune_rule=2, ext_min_n=0), dict(prune_rule=2, ext_min_n=3, ext_thr=float("nan")),
                dict(prune_rule=4, hist_min_n=0, hist_min_arms=3),
                dict(prune_rule=4, hist_min_n=6, hist_min_arms=3, hist_kappa=-1.0),
                dict(prune_rule=8, cascade_k=17),
                dict(exploit=2), dict(exploit=1, ph_lambda=-1.0), dict(exploit=1, ph_delta=float("nan")),
                dict(exploit=1, ph_window=-1), dict(exploit=1, ph_min_rounds=-5),
                dict(refine=2), dict(refine=1, refine_period=0, refine_stride=10, refine_min_n=4),
                dict(refine=1, refine_period=50, refine_stride=0, refine_min_n=4),
                dict(refine=1, refine_period=50, refine_stride=10, refine_half=-1, refine_min_n=4),
                dict(refine=1, refine_period=50, refine_stride=10, refine_min_n=0)):
        assert L.agft_state_bytes(_cfg(**bad)) == 0, bad


def test_state_bytes_with_exploitation(lib):
    """The switch adds the contiguous theta copy, B*K*d floats."""
    ph = dict(ph_delta=0.05, ph_lambda=5.0, ph_window=100, ph_min_rounds=100)
    for B, K, d in ((4, 16, 8), (1000, 128, 16), (3, 1024, 32)):
        off = L.agft_state_bytes(_cfg(B=B, K=K, d=d, **ph))
        on = L.agft_state_bytes(_cfg(B=B, K=K, d=d, exploit=1, **ph))
        copy = B * K * d * 4
        assert copy <= on - off < copy + 256 and on % 256 == 0


def test_create_rejects_before_launch(lib):
    cfg = _cfg()
    n = L.agft_state_bytes(cfg)
    code, h = L.agft_create(cfg, None, n, None)
    assert code == L.AGFT_E_INVAL and not h.value
    code, h = L.agft_create(cfg, ctypes.c_void_p(0x1001), n, None)   # misaligned
    assert code == L.AGFT_E_INVAL
    code, h = L.agft_create(cfg, ctypes.c_void_p(0x100000), n - 1, None)  # too small
    assert code == L.AGFT_E_INVAL
    code, h = L.agft_create(_cfg(d=12), ctypes.c_void_p(0x100000), 1 << 30, None)
    assert code == L.AGFT_E_UNSUPPORTED
    # a non-sticky rule 1 is built for rule 1 alone
    heur = dict(ext_rounds=60, ext_min_n=3, ext_thr=-1.2)
    code, h = L.agft_create(_cfg(prune_rule=3, prune_sticky=0, **heur), ctypes.c_void_p(0x100000),
                            1 << 30, None)
    assert code == L.AGFT_E_UNSUPPORTED
    assert L.agft_state_bytes(_cfg(prune_rule=1, prune_sticky=0)) == n
    code, shape = L.agft_launch_shape_for(_cfg(prune_rule=3, prune_sticky=0, **heur))
    assert code == L.AGFT_E_UNSUPPORTED
    code, h = L.agft_create(_cfg(alpha0=-1.0), ctypes.c_void_p(0x100000), 1 << 30, None)
    assert code == L.AGFT_E_INVAL
    assert lib.agft_create(ctypes.byref(cfg), ctypes.c_void_p(0x100000), n, None, None) == L.AGFT_E_INVAL


def test_null_handle_calls(lib):
    assert L.agft_step(None, None, None, None, None) == L.AGFT_E_INVAL
    code, _ = L.agft_get_state(None)
    assert code == L.AGFT_E_INVAL
    assert L.agft_export(None, None, None) == L.AGFT_E_INVAL
    assert L.agft_set_stream(None, None) == L.AGFT_E_INVAL
    assert L.agft_destroy(None) == L.AGFT_OK


def _env_cfg(**kw):
    from agft_workloads import ENV, get_workload
    from paper_2508_01744_amd.env import env_config
    cfg = env_config(get_workload(2, B=8, T=10), ENV)
    for k, v in kw.items():
        setattr(cfg, k, v)
    return cfg


def test_env_validation(lib):
    assert L.agft_env_state_bytes(_env_cfg()) > 0
    for bad in (dict(B=0), dict(K=0), dict(d=7), dict(T=0), dict(lat_min=0.0), dict(f_lo=0.0),
                dict(tpot_div=0.0), dict(svc_lo=0), dict(q_cap=-1)):
        assert L.agft_env_state_bytes(_env_cfg(**bad)) == 0, bad
    cfg = _env_cfg()
    n = L.agft_env_state_bytes(cfg)
    p = ctypes.c_void_p(0x100000)
    assert L.agft_env_reset(cfg, None, n, p, p, p, None) == L.AGFT_E_INVAL
    assert L.agft_env_reset(cfg, ctypes.c_void_p(0x1001), n, p, p, p, None) == L.AGFT_E_INVAL
    assert L.agft_env_reset(cfg, p, n - 1, p, p, p, None) == L.AGFT_E_INVAL
    assert L.agft_env_step(cfg, p, n, -1, p, p, p, p, p, None) == L.AGFT_E_INVAL
    assert L.agft_env_step(cfg, p, n, cfg.T, p, p, p, p, p, None) == L.AGFT_E_INVAL
    assert L.agft_env_step(cfg, p, n, 0, None, p, p, p, p, None) == L.AGFT_E_INVAL
    # contexts leave as float4 stores: a context buffer off 16 bytes is refused
    q = ctypes.c_void_p(0x100008)
    assert L.agft_env_reset(cfg, p, n, p, p, q, None) == L.AGFT_E_INVAL
    assert L.agft_env_step(cfg, p, n, 0, p, p, p, p, q, None) == L.AGFT_E_INVAL


def test_sim_step_rejects_before_launch(lib):
    """agft_sim_step checks its arguments before anything is enqueued: no
    handle, a missing buffer, an environment of another shape."""
    cfg = _env_cfg()
    n = L.agft_env_state_bytes(cfg)
    p = ctypes.c_void_p(0x100000)
    assert L.agft_sim_step(None, cfg, p, n, p, p, p, p, p, None) == L.AGFT_E_INVAL
    bad = _env_cfg(d=7)
    assert L.agft_sim_step(None, bad, p, n, p, p, p, p, p, None) == L.AGFT_E_INVAL


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    """No silent fallback: without the built library every entry point raises."""
    monkeypatch.setattr(L, "LIB_PATH", str(tmp_path / "libagft.so"))
    monkeypatch.setattr(L, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        L.lib()
    with pytest.raises(RuntimeError):
        L.agft_abi_version()
