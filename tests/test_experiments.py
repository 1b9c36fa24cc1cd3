"""The quality-experiment helpers (CPU): the noise-free EDP used for the
offline optimum and the window metrics decoded from the environment's
context, pinned to the fp64 environment model; the per-instance mean and
coefficient of variation against numpy."""
import numpy as np
import torch

from agft_workloads import ENV, exogenous, get_workload
from oracle.env import Env
from paper_2508_01744_amd import experiments as E


def _const_run(wl, arm, T):
    arr, noi = exogenous(wl, T=T)
    env = Env(wl, arr, np.zeros_like(noi), T)
    x = env.reset()
    rs, xs = [], []
    for t in range(T):
        r, x = env.step(t, np.full(env.n, arm, dtype=np.int64))
        rs.append(r.copy())
        xs.append(x.copy())
    return arr, np.array(rs), np.array(xs)


def test_noise_free_edp_ranks_arms_like_the_environment():
    """With no noise the environment's reward is -EDP / EDP_ref with EDP_ref
    independent of the arm, so reward ratios between arms are EDP ratios."""
    T = 40
    wl = get_workload("cfg5", B=6, K=9, T=T)       # drifting b, c
    runs = [_const_run(wl, k, T) for k in range(wl.K)]
    arr = runs[0][0]
    clocks = E.arm_clocks(wl.K, "cpu")
    for t in (0, 17, T - 1):
        n = torch.as_tensor(arr[t + 1], dtype=torch.float64)[:, None]
        edp = E.noise_free_edp(n, clocks[None, :], E.drift_scale(wl, t)).numpy()
        rew = np.stack([runs[k][1][t] for k in range(wl.K)], axis=1)
        np.testing.assert_allclose(edp / edp[:, -1:], rew / rew[:, -1:], rtol=1e-12)
        assert (edp.argmin(axis=1) == rew.argmax(axis=1)).all()


def test_window_metrics_from_context():
    """At the top clock with no noise the reward is exactly -1, i.e. the
    window's EDP equals the closed form at f = 1; the metrics decoded from
    the context must reproduce it."""
    T = 30
    wl = get_workload("cfg3", B=5, T=T)
    arr, rs, xs = _const_run(wl, wl.K - 1, T)
    assert np.allclose(rs, -1.0)
    for t in (0, 11, T - 1):
        m = E.window_metrics(torch.as_tensor(xs[t]), torch.tensor(ENV["f_hi"], dtype=torch.float64),
                             E.drift_scale(wl, t))
        n = torch.as_tensor(arr[t + 1], dtype=torch.float64)[:, None]
        ref = E.noise_free_edp(n, torch.tensor([ENV["f_hi"]], dtype=torch.float64), E.drift_scale(wl, t))
        np.testing.assert_allclose(m["edp"].numpy(), ref[:, 0].numpy(), rtol=1e-9)
        np.testing.assert_allclose(m["edp"].numpy(), (m["energy"] * m["tpot"] * ENV["tpot_div"]).numpy())


def test_accumulator_mean_and_cv():
    rng = np.random.default_rng(0)
    B, T = 7, 50
    vals = {m: rng.uniform(0.5, 2.0, size=(T, B)) for m in E.METRICS}
    mask = rng.uniform(size=(T, B)) < 0.6
    acc = E._Acc(B, "cpu")
    for t in range(T):
        acc.add({m: torch.as_tensor(vals[m][t]) for m in E.METRICS}, torch.as_tensor(mask[t]))
    out = acc.summary()
    for m in E.METRICS:
        means, cvs = [], []
        for i in range(B):
            v = vals[m][mask[:, i], i]
            means.append(v.mean())
            cvs.append(v.std() / v.mean())
        assert abs(out[m]["mean"] - np.mean(means)) < 1e-12
        assert abs(out[m]["cv"] - np.mean(cvs)) < 1e-9
