"""Closed-loop batched simulation on one GPU: the environment kernel and the
tuner step kernel alternate on one stream."""
import torch

from .env import GpuEnv, env_config
from .tuner import Tuner


def run_closed_loop(wl, env_constants, arrivals, noise, T=None, probes=None, scores=False,
                    device="cuda", fused=False):
    """Run T decisions of wl.B instances.

    arrivals, noise: [T+1][B] (numpy or torch) exogenous draws.
    fused: each decision and the environment's response through
    agft_sim_step (one launch up to 8,192 instances) instead of agft_step
    and agft_env_step.
    probes: instance indices to record at every step (contexts, rewards,
    actions, masks, test words, action spaces; with scores, the scores and
    the top-two gap of each decision); the records are returned as host
    tensors.
    """
    T = wl.T if T is None else int(T)
    dev = torch.device(device)
    arr = torch.as_tensor(arrivals, dtype=torch.int32).to(dev)
    noi = torch.as_tensor(noise, dtype=torch.float32).to(dev)
    env = GpuEnv(env_config(wl, env_constants, T=T), arr, noi)
    tuner = Tuner.from_workload(wl, device=dev)
    action = torch.empty(wl.B, dtype=torch.int32, device=dev)
    sc = torch.empty(wl.B, 2, wl.K, device=dev) if scores else None
    rec = None
    if probes is not None:
        pidx = torch.as_tensor(list(probes), dtype=torch.long, device=dev)
        P = pidx.numel()
        rec = dict(x=torch.empty(T, P, wl.d, device=dev),
                   r=torch.empty(T, P, device=dev),
                   a=torch.empty(T, P, dtype=torch.int32, device=dev),
                   mask=torch.empty(T, P, (wl.K + 31) // 32, dtype=torch.int32, device=dev),
                   kact=torch.empty(T, P, dtype=torch.int32, device=dev),
                   ph=torch.empty(T, P, 9, dtype=torch.int32, device=dev),
                   win=torch.empty(T, P, 3, dtype=torch.int32, device=dev))
        if scores:
            rec["scores"] = torch.empty(T, P, 2, wl.K, device=dev)
            rec["gap"] = torch.empty(T, P, device=dev)
        view = tuner.view()
    x = env.reset()
    r = None
    for t in range(T):
        if rec is not None:
            rec["x"][t] = x.index_select(0, pidx)
        if fused:
            r, x = env.fused_step(tuner, action, sc)
        else:
            tuner.step(x, r, action, sc)
        if rec is not None:
            rec["a"][t] = action.index_select(0, pidx)
            rec["mask"][t] = view["mask"].index_select(0, pidx)
            rec["kact"][t] = view["kact"].index_select(0, pidx)
            rec["ph"][t] = view["ph"].index_select(0, pidx)
            rec["win"][t] = view["window"].index_select(0, pidx)
            if scores:
                rec["scores"][t] = sc.index_select(0, pidx)
                rec["gap"][t] = view["gap"].index_select(0, pidx)
        if not fused:
            r, x = env.step(t, action)
        if rec is not None:
            rec["r"][t] = r.index_select(0, pidx)
    tuner.flush(r)
    out = dict(tuner=tuner, env=env, last_action=action)
    if rec is not None:
        torch.cuda.synchronize(dev)
        out["probes"] = {k: v.cpu() for k, v in rec.items()}
    return out
