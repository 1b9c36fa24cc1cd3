"""The simulator's fused step (agft_sim_step: the decision and the
environment's response in one launch, up to 8,192 instances) against the two
separate calls it replaces, and against the oracle.

Fused and separate runs of the same workload must agree bit for bit:
contexts, rewards, actions, masks, scores, top-two gaps and the final state
buffer.  Full-size fused runs of the two workloads where the second launch
weighs most (cfg1, cfg2) are also checked against the fp64 oracle and its
environment like the separate runs."""
import ctypes

import pytest
import torch

import parity
import paper_2508_01744_amd._lib as L
from agft_workloads import ENV, exogenous, get_workload, probe_instances
from gpu_helpers import say
from paper_2508_01744_amd import AgftError, GpuEnv, Tuner, env_config, run_closed_loop

pytestmark = pytest.mark.gpu

SMALL = {"cfg1": dict(T=600), "cfg2": dict(B=48, T=300), "cfg3": dict(B=24, T=200),
         "cfg4": dict(B=40, T=200), "cfg5": dict(B=12, T=300), "cfg2per": dict(B=32, T=300),
         "cfg4pe": dict(B=24, T=260), "cfg5n": dict(B=8, T=200), "cfg3r": dict(B=16, T=200)}


@pytest.mark.parametrize("name", list(SMALL))
def test_fused_equals_separate(name):
    wl = get_workload(name, **SMALL[name])
    say(f"[fused] {wl.name} B={wl.B} K={wl.K} d={wl.d} T={wl.T}")
    arr, noi = exogenous(wl)
    ids = list(range(wl.B))
    sep = run_closed_loop(wl, ENV, arr, noi, probes=ids, scores=True)
    fus = run_closed_loop(wl, ENV, arr, noi, probes=ids, scores=True, fused=True)
    for key in sep["probes"]:
        a, b = sep["probes"][key], fus["probes"][key]
        assert torch.equal(a.view(torch.int32) if a.is_floating_point() else a,
                           b.view(torch.int32) if b.is_floating_point() else b), key
    assert torch.equal(sep["tuner"].state, fus["tuner"].state)
    assert torch.equal(sep["env"].state, fus["env"].state)


def test_large_batch_simulator_step_equals_separate():
    """Above 8,192 instances agft_sim_step runs the step kernel and then the
    environment kernel: the same results as the separate calls, bit for bit,
    and the same in-place buffers (one instance past the threshold)."""
    wl = get_workload("cfg3", B=8193, T=40)
    say(f"[fused] two launches: {wl.name} B={wl.B} K={wl.K} d={wl.d} T={wl.T}")
    arr, noi = exogenous(wl)
    ids = [0, 1, 4096, 8191, 8192]
    sep = run_closed_loop(wl, ENV, arr, noi, probes=ids, scores=True)
    fus = run_closed_loop(wl, ENV, arr, noi, probes=ids, scores=True, fused=True)
    for key in sep["probes"]:
        a, b = sep["probes"][key], fus["probes"][key]
        assert torch.equal(a.view(torch.int32) if a.is_floating_point() else a,
                           b.view(torch.int32) if b.is_floating_point() else b), key
    assert torch.equal(sep["tuner"].state, fus["tuner"].state)
    assert torch.equal(sep["env"].state, fus["env"].state)


@pytest.mark.parametrize("name", ["cfg1", "cfg2"])
def test_fused_full_size_parity(name):
    wl = get_workload(name)
    probes = probe_instances(wl.B, 64)
    say(f"[fused] parity {wl.name} B={wl.B} T={wl.T} probes={len(probes)}")
    arr, noi = exogenous(wl)
    out = run_closed_loop(wl, ENV, arr, noi, probes=probes, scores=True, fused=True)
    st = parity.compare(wl, wl.T, probes, out["probes"])
    say(f"[fused] {wl.name}: max score err {st['max_score_err']:.2e}, ctx err {st['max_ctx_err']:.2e}, "
        f"reward err {st['max_reward_err']:.2e}, forced {st['forced']}/{st['decisions']}")


def test_fused_step_errors():
    """Past the last window of the draws the fused step is refused; so is an
    environment of another shape."""
    wl = get_workload(2, B=8, T=3)
    dev = torch.device("cuda")
    arr, noi = exogenous(wl)
    env = GpuEnv(env_config(wl, ENV), torch.as_tensor(arr, device=dev), torch.as_tensor(noi, device=dev))
    tun = Tuner.from_workload(wl, device=dev)
    act = torch.empty(wl.B, dtype=torch.int32, device=dev)
    env.reset()
    for _ in range(wl.T):
        env.fused_step(tun, act)
    with pytest.raises(AgftError) as e:
        env.fused_step(tun, act)
    assert e.value.code == L.AGFT_E_STATE
    other = Tuner(wl.B + 1, wl.K, wl.d, device=dev)
    vp = lambda t: ctypes.c_void_p(t.data_ptr())
    code = L.agft_sim_step(other.h, env.cfg, vp(env.state), env.nbytes, vp(env.arrivals), vp(env.noise),
                           vp(env.ctx), vp(env.reward), vp(act), None)
    assert code == L.AGFT_E_INVAL
    torch.cuda.synchronize()
