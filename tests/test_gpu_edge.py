"""Edge cases of the GPU step against the oracle (open loop: the same given
contexts and rewards to both sides), plus API semantics: flush, missing
reward, non-finite inputs, resume from a saved buffer, determinism."""
import numpy as np
import pytest
import torch

import parity
import paper_2508_01744_amd._lib as L
from agft_workloads import ENV, exogenous, get_workload
from gpu_helpers import compare_model, random_contexts, run_open_loop, say
from paper_2508_01744_amd import AgftError, Tuner, run_closed_loop

pytestmark = pytest.mark.gpu


def _cfg(B, K, d, lam=1.0, alpha0=0.5, sched=0, prune=0, period=50):
    return dict(B=B, K=K, d=d, lam=lam, alpha0=alpha0, sched=sched, prune=prune, period=period,
                heuristics=None)


def _open_loop_case(name, cfg, T, seed, scale=1.0):
    say(f"[edge] {name}: {cfg} T={T}")
    X, R = random_contexts(seed, T, cfg["B"], cfg["d"], scale)
    a, m, s, tuner, _ = run_open_loop(cfg, X, R)
    st = parity.compare_open_loop(name, cfg, X, R, a, m, s)
    compare_model(tuner, st["oracle"], range(cfg["B"]), 1e-3, 1e-4)
    say(f"[edge] {name}: max score err {st['max_score_err']:.2e}, forced {st['forced']}/"
        f"{st['decisions']}, exact-tie steps {st['exact_tie_steps']}")
    return st, a, tuner


@pytest.mark.parametrize("d", [8, 16, 32])
def test_single_arm(d):
    st, a, _ = _open_loop_case(f"K=1 d={d}", _cfg(3, 1, d), 40, 1)
    assert (a == 0).all()


@pytest.mark.parametrize("d,T", [(8, 60), (16, 50), (32, 40)])
def test_max_arms(d, T):
    """K = 1024, the largest arm count: 2.3 MB of records per instance at d = 32."""
    _open_loop_case(f"K=1024 d={d}", _cfg(3, 1024, d, prune=1, period=20), T, 2)


@pytest.mark.parametrize("K", [63, 65, 100, 129, 255])
def test_ragged_arm_counts(K):
    _open_loop_case(f"K={K} d=16", _cfg(5, K, 16, alpha0=0.3, prune=1, period=10), 120, K)


def test_greedy_alpha_zero_with_pruning():
    st, a, tuner = _open_loop_case("alpha=0", _cfg(6, 40, 8, alpha0=0.0, prune=1, period=15), 60, 3)
    # alpha = 0: UCB = LCB, so each prune keeps only arms tied with the best estimate
    kact = tuner.view()["kact"].cpu().numpy()
    assert (kact >= 1).all()


def test_decaying_alpha_d32():
    _open_loop_case("alpha0/sqrt(t+1) d=32", _cfg(4, 70, 32, alpha0=1.0, sched=1, prune=1,
                                                    period=25), 150, 4)


def test_untouched_arms_are_swept_in_order():
    """All-untouched arms tie exactly; the GPU must break ties to the lowest
    index, so constant contexts and negative rewards sweep arms 0..K-1."""
    K, B, d = 70, 2, 16
    cfg = _cfg(B, K, d, alpha0=1.0)
    X = np.zeros((K, B, d))
    X[:, :, 0] = 1.0
    X[:, :, 1:] = np.random.default_rng(5).standard_normal((1, B, d - 1)).astype(np.float32)
    R = -np.ones((K, B))
    a, m, s, tuner, _ = run_open_loop(cfg, X, R)
    assert (a == np.arange(K)[:, None]).all()


RULES = dict(ext_rounds=60, ext_min_n=3, ext_thr=-1.2, hist_after=30, hist_min_n=6, hist_kappa=1.0,
             hist_min_arms=3, cascade_k=0)


def test_missing_reward_and_flush():
    dev = torch.device("cuda")
    # rule bit 4 on, so that the per-arm reward statistics are kept
    tuner = Tuner(4, 16, 8, prune_rule=4, device=dev, heuristics=RULES)
    X, R = random_contexts(6, 3, 4, 8)
    x = torch.as_tensor(X, dtype=torch.float32, device=dev)
    r = torch.as_tensor(R, dtype=torch.float32, device=dev)
    tuner.step(x[0])
    with pytest.raises(AgftError) as e:
        tuner.step(x[1])
    assert e.value.code == L.AGFT_E_STATE
    tuner.step(x[1], r[0])
    tuner.flush(r[1])
    v = tuner.view()
    torch.cuda.synchronize()
    assert int(v["stats"][..., 0].sum()) == 8 and v["pending"] == 0
    assert (v["aprev"].cpu() == -1).all()
    tuner.step(x[2])          # no reward needed after a flush
    torch.cuda.synchronize()
    assert tuner.t == 3


def test_statistics_only_kept_when_read():
    """Without rules 2-8 or the refinement nothing reads the per-arm reward
    statistics: they stay zero, and a buffer made so cannot be adopted by a
    configuration that reads them."""
    dev = torch.device("cuda")
    X, R = random_contexts(7, 3, 4, 8)
    x = torch.as_tensor(X, dtype=torch.float32, device=dev)
    r = torch.as_tensor(R, dtype=torch.float32, device=dev)
    tuner = Tuner(4, 16, 8, device=dev)
    tuner.step(x[0])
    tuner.step(x[1], r[0])
    tuner.flush(r[1])
    torch.cuda.synchronize()
    assert int(tuner.view()["stats"].abs().sum()) == 0
    state = tuner.state.clone()
    tuner.close()
    with pytest.raises(AgftError) as e:
        Tuner(4, 16, 8, prune_rule=4, device=dev, heuristics=RULES, state=state, adopt=True)
    assert e.value.code == L.AGFT_E_STATE


def test_non_finite_inputs():
    """NaN reward: that update is skipped; NaN or inf in a context: no
    decision (-1) and no update next step; both counted; oracle agrees."""
    cfg = _cfg(6, 20, 8, prune=1, period=7)
    T = 40
    X, R = random_contexts(7, T, 6, 8)
    R[5, 1] = np.nan
    R[9, 2] = np.inf
    X[12, 3, 4] = np.nan
    X[13, 3, 2] = np.inf
    X[20, 0, 0] = -np.inf
    a, m, s, tuner, _ = run_open_loop(cfg, X, R)
    st = parity.compare_open_loop("non-finite", cfg, X, R, a, m, s)
    assert a[12, 3] == -1 and a[13, 3] == -1 and a[20, 0] == -1
    bad = tuner.view()["bad"].cpu().numpy()
    ora_bad = [st["oracle"].get(i)["bad"] for i in range(6)]
    assert list(bad) == ora_bad
    assert bad[1] == 1 and bad[2] == 1 and bad[3] == 2 and bad[0] == 1
    compare_model(tuner, st["oracle"], range(6), 1e-3, 1e-4)


def test_resume_from_saved_buffer_is_bit_identical():
    wl = get_workload(4, B=64, T=120)
    arr, noi = exogenous(wl)
    dev = torch.device("cuda")
    full = run_closed_loop(wl, ENV, arr, noi, probes=range(wl.B))
    # the same run, interrupted after T1 decisions: copy the buffer, adopt it
    from paper_2508_01744_amd import GpuEnv, env_config
    T1 = 53
    env = GpuEnv(env_config(wl, ENV), torch.as_tensor(arr, device=dev),
                 torch.as_tensor(noi, device=dev))
    t1 = Tuner.from_workload(wl, device=dev)
    act = torch.empty(wl.B, dtype=torch.int32, device=dev)
    x = env.reset()
    r = None
    acts = []
    for t in range(wl.T):
        if t == T1:
            saved = t1.state.clone()
            t1.close()
            t1 = Tuner.from_workload(wl, device=dev, state=saved, adopt=True)
            assert t1.t == T1
        t1.step(x, r, act)
        acts.append(act.clone())
        r, x = env.step(t, act)
    t1.flush(r)
    torch.cuda.synchronize()
    acts = torch.stack(acts).cpu()
    assert torch.equal(acts, full["probes"]["a"])
    assert torch.equal(t1.state, full["tuner"].state)


def test_adopt_rejects_mismatched_buffer():
    dev = torch.device("cuda")
    t1 = Tuner(8, 16, 8, device=dev)
    torch.cuda.synchronize()
    with pytest.raises(AgftError) as e:
        Tuner(8, 32, 8, device=dev, state=t1.state.clone(), adopt=True)   # too small for K=32
    assert e.value.code == L.AGFT_E_INVAL
    with pytest.raises(AgftError) as e:
        Tuner(8, 16, 8, device=dev, state=torch.zeros_like(t1.state), adopt=True)  # no header
    assert e.value.code == L.AGFT_E_STATE
    big = torch.zeros(Tuner(8, 16, 16, device=dev).nbytes, dtype=torch.uint8, device=dev)
    big[: t1.state.numel()].copy_(t1.state)
    with pytest.raises(AgftError) as e:
        Tuner(8, 16, 16, device=dev, state=big, adopt=True)   # header says d = 8
    assert e.value.code == L.AGFT_E_STATE
    t2 = Tuner(8, 16, 8, device=dev, state=t1.state.clone(), adopt=True)
    assert t2.t == 0


def test_determinism():
    wl = get_workload(5, B=16, T=150)
    arr, noi = exogenous(wl)
    a = run_closed_loop(wl, ENV, arr, noi, probes=range(wl.B), scores=True)
    b = run_closed_loop(wl, ENV, arr, noi, probes=range(wl.B), scores=True)
    for key in a["probes"]:
        assert torch.equal(a["probes"][key], b["probes"][key]), key
    assert torch.equal(a["tuner"].state, b["tuner"].state)


AGGRESSIVE = dict(ext_rounds=40, ext_min_n=1, ext_thr=-1.0, hist_after=10, hist_min_n=2,
                  hist_kappa=0.5, hist_min_arms=3)


@pytest.mark.parametrize("d,K,rules", [(8, 20, 2 | 8), (16, 70, 4), (16, 40, 15), (32, 33, 14),
                                       (8, 1024, 15)])
def test_paper_pruning_rules(d, K, rules):
    """The paper's extreme/historical/cascade rules (Sec. 4.3) with thresholds
    set so that they fire often, against the oracle (open loop)."""
    cfg = _cfg(6, K, d, alpha0=0.6, prune=rules, period=25)
    cfg["heuristics"] = dict(AGGRESSIVE, cascade_k=K // 2)
    T = 120 if K < 1024 else 60
    st, a, tuner = _open_loop_case(f"rules={rules} d={d} K={K}", cfg, T, 100 + K)
    kact = tuner.view()["kact"].cpu().numpy()
    assert (kact >= 1).all() and (kact < K).any()
    say(f"[edge] rules forced {st['forced_rules']}")


def test_side_stream_and_stream_switch():
    """The same closed-loop run enqueued on a side stream (default priority),
    moved back to the default stream halfway, ends in a bit-identical state."""
    from paper_2508_01744_amd import GpuEnv, env_config
    wl = get_workload(3, B=32, T=120)
    arr, noi = exogenous(wl)
    ref = run_closed_loop(wl, ENV, arr, noi, probes=range(wl.B))
    dev = torch.device("cuda")
    main = torch.cuda.current_stream(dev)
    side = torch.cuda.Stream(device=dev)
    side.wait_stream(main)
    with torch.cuda.stream(side):
        arr_d, noi_d = torch.as_tensor(arr, device=dev), torch.as_tensor(noi, device=dev)
        env = GpuEnv(env_config(wl, ENV), arr_d, noi_d, stream=side)
        tun = Tuner.from_workload(wl, device=dev, stream=side)
        act = torch.empty(wl.B, dtype=torch.int32, device=dev)
        x, r, acts = env.reset(), None, []
        for t in range(60):
            tun.step(x, r, act)
            acts.append(act.clone())
            r, x = env.step(t, act)
    main.wait_stream(side)
    tun.set_stream(main)
    env.stream = main
    for t in range(60, wl.T):
        tun.step(x, r, act)
        acts.append(act.clone())
        r, x = env.step(t, act)
    tun.flush(r)
    torch.cuda.synchronize()
    assert torch.equal(torch.stack(acts).cpu(), ref["probes"]["a"])
    assert torch.equal(tun.state, ref["tuner"].state)
