"""The fp64 environment model against closed forms and invariants (CPU only).

The environment's constants are chosen here (the paper prints no worked
example of its reward or features), so only its structure is pinned here:
the energy-delay product's defining identities and the position of its
optimum, the integer service capacities, and the context layout.
"""
import numpy as np

from agft_workloads import ENV, get_workload, exogenous
from oracle import Env


def _env(cfg, n, T, arrivals=None, noise=None, **over):
    wl = get_workload(cfg, B=n, T=T, **over)
    if arrivals is None:
        arrivals, noise = exogenous(wl)
    return wl, Env(wl, arrivals, noise, T)


def test_power_and_reference_reward():
    """power(1) = 1, and without noise the full clock earns reward -1 (its EDP
    is the reference EDP), with or without coefficient drift."""
    assert ENV["P0"] + ENV["c"] == 1.0
    for drift in (0.0, 0.3):
        T, n = 30, 4
        arrivals = np.random.default_rng(0).integers(0, 30, size=(T + 1, n)).astype(np.int32)
        noise = np.zeros((T + 1, n), dtype=np.float32)
        wl, env = _env(2, n, T, arrivals, noise, K=64, drift=drift)
        env.reset()
        for t in range(T):
            r, _ = env.step(t, np.full(n, wl.K - 1))
            assert np.allclose(r, -1.0, rtol=0, atol=1e-15)


def test_edp_optimum_solves_stationarity():
    """Noise-free EDP(f) = (P0 + c f^3)(a + b n / f)^2 is smallest where
    3 a c f^4 + b n c f^3 - 2 b n P0 = 0 (derivative set to zero); the
    best-rewarded arm on a fine grid sits within one grid step of that root,
    and the root moves up with load (the U-shape of Fig. 6)."""
    K = 1025
    roots = []
    for load in (1, 3, 6, 10, 15, 20, 28):
        T = 1
        arrivals = np.full((T + 1, K), load, dtype=np.int32)
        noise = np.zeros((T + 1, K), dtype=np.float32)
        wl, env = _env(2, K, T, arrivals, noise, K=K)
        env.reset()
        r, _ = env.step(0, np.arange(K))
        f_best = env.arm_clock(int(np.argmax(r)))
        a, b, c, P0 = ENV["a"], ENV["b"], ENV["c"], ENV["P0"]
        poly = np.roots([3 * a * c, b * load * c, 0.0, 0.0, -2 * b * load * P0])
        root = [z.real for z in poly if abs(z.imag) < 1e-12 and z.real > 0][0]
        root = min(max(root, ENV["f_lo"]), ENV["f_hi"])
        assert abs(f_best - root) <= (ENV["f_hi"] - ENV["f_lo"]) / (K - 1)
        roots.append(root)
    assert all(x < y for x, y in zip(roots, roots[1:]))
    assert ENV["f_lo"] < roots[0] < roots[-1] < ENV["f_hi"]


def test_integer_capacities_by_hand():
    wl, env = _env(2, 1, 5, K=5)
    assert list(env.arm_capacity(np.arange(5))) == [5, 10, 15, 20, 25]
    wl, env = _env(2, 1, 5, K=16)
    # round(5 + 4k/3), worked by hand
    assert list(env.arm_capacity(np.arange(16))) == [5, 6, 8, 9, 10, 12, 13, 14, 16, 17,
                                                      18, 20, 21, 22, 24, 25]
    wl, env = _env(2, 1, 5, K=1)
    assert list(env.arm_capacity(np.arange(1))) == [25]


def test_context_layout_and_lags():
    """Bias first; lagged feature blocks are the previous contexts' blocks;
    the reward slots hold the rewards of the latest decisions; windows before
    the warm-up repeat it."""
    T = 40
    for d, cfg in ((8, 2), (16, 3), (32, 5)):
        wl, env = _env(cfg, 6, T)
        rng = np.random.default_rng(d)
        x = env.reset()
        assert np.all(x[:, 0] == 1.0)
        if d >= 16:
            assert np.array_equal(x[:, 8:15], x[:, 1:8])
        xs, rs = [x], []
        for t in range(T):
            r, x = env.step(t, rng.integers(0, wl.K, size=6))
            xs.append(x)
            rs.append(r)
        for t in range(1, T + 1):
            cur, prev = xs[t], xs[t - 1]
            assert np.all(cur[:, 0] == 1.0)
            if d == 16:
                assert np.array_equal(cur[:, 8:15], prev[:, 1:8])
                assert np.array_equal(cur[:, 15], rs[t - 1])
            if d == 32:
                assert np.array_equal(cur[:, 8:15], prev[:, 1:8])
                assert np.array_equal(cur[:, 15:22], prev[:, 8:15])
                assert np.array_equal(cur[:, 22:29], prev[:, 15:22])
                assert np.array_equal(cur[:, 29], rs[t - 1])
                assert np.array_equal(cur[:, 30:32], prev[:, 29:31])


def test_raw_feature_ranges():
    """Decoded features respect the caps: queue in [0, q_cap], running <=
    run_cap, util <= 1, clock equals the chosen arm's value."""
    T, n = 300, 32
    wl, env = _env(4, n, T)
    mu, sd = np.array(ENV["mu"]), np.array(ENV["sd"])
    rng = np.random.default_rng(3)
    env.reset()
    for t in range(T):
        a = rng.integers(0, wl.K, size=n)
        _, x = env.step(t, a)
        raw = x[:, 1:8] * sd + mu
        q = np.expm1(raw[:, 1])
        assert np.all(q > -1e-9) and np.all(q <= ENV["q_cap"] + 1e-9)
        assert np.all(np.abs(q - np.round(q)) < 1e-9)
        assert np.all(raw[:, 2] <= ENV["run_cap"] + 1e-9)
        assert np.all(raw[:, 5] <= 1.0 + 1e-12)
        assert np.allclose(raw[:, 6], env.arm_clock(a), rtol=0, atol=1e-12)
