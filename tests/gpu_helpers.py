"""GPU-side drivers shared by the GPU tests (they call the C ABI through the
package binding; nothing here computes the method)."""
import sys

import numpy as np
import torch

from paper_2508_01744_amd import Tuner


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run_open_loop(cfg, X, R, flush=True):
    """Drive a Tuner with given contexts X [T][B][d] and rewards R [T][B].
    Returns host arrays: actions [T][B], mask words [T][B][KW], scores
    [T][B][2][K], the tuner, and a dict of the Page-Hinkley words [T][B][9]
    ("ph"), the action spaces [T][B][3] ("win") and the top-two gaps [T][B]
    ("gap") after each step."""
    T, B, d = X.shape
    dev = torch.device("cuda")
    tuner = Tuner(cfg["B"], cfg["K"], cfg["d"], cfg["lam"], cfg["alpha0"], cfg["sched"],
                  cfg["prune"], cfg["period"], device=dev, heuristics=cfg.get("heuristics"),
                  exploit=cfg.get("exploit"), refine=cfg.get("refine"),
                  prune_sticky=cfg.get("sticky", 1))
    Xd = torch.as_tensor(np.asarray(X, dtype=np.float32), device=dev)
    Rd = torch.as_tensor(np.asarray(R, dtype=np.float32), device=dev)
    K, KW = cfg["K"], (cfg["K"] + 31) // 32
    acts = torch.empty(T, B, dtype=torch.int32, device=dev)
    masks = torch.empty(T, B, KW, dtype=torch.int32, device=dev)
    scores = torch.empty(T, B, 2, K, device=dev)
    ph = torch.empty(T, B, 9, dtype=torch.int32, device=dev)
    win = torch.empty(T, B, 3, dtype=torch.int32, device=dev)
    gap = torch.empty(T, B, device=dev)
    view = tuner.view()
    for t in range(T):
        tuner.step(Xd[t], Rd[t - 1] if t > 0 else None, acts[t], scores[t])
        masks[t].copy_(view["mask"])
        ph[t].copy_(view["ph"])
        win[t].copy_(view["window"])
        gap[t].copy_(view["gap"])
    if flush and T > 0:
        tuner.flush(Rd[T - 1])
    torch.cuda.synchronize()
    return (acts.cpu().numpy(), masks.cpu().numpy(), scores.cpu().numpy().astype(np.float64), tuner,
            dict(ph=ph.cpu().numpy(), win=win.cpu().numpy(), gap=gap.cpu().numpy().astype(np.float64)))


def random_contexts(seed, T, B, d, scale=1.0):
    """Bias plus standard-normal features (test inputs, same arrays to both sides)."""
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((T, B, d)) * scale
    X[:, :, 0] = 1.0
    R = rng.uniform(-2.0, 0.0, size=(T, B))
    return X.astype(np.float32).astype(np.float64), R.astype(np.float32).astype(np.float64)


def compare_model(tuner, ora, ids, theta_tol, ainv_tol):
    """Final theta and A^{-1} of the GPU model vs the oracle's, for instances ids."""
    th, ai = tuner.export(theta=True, ainv=True)
    th = th.cpu().numpy().astype(np.float64)
    ai = ai.cpu().numpy().astype(np.float64)
    worst_th = worst_ai = 0.0
    for row, i in enumerate(ids):
        st = ora.get(row)
        e_th = np.abs(th[i] - st["theta"]).max() / max(1.0, np.abs(st["theta"]).max())
        e_ai = np.abs(ai[i] - st["Ainv"]).max() / max(1.0, np.abs(st["Ainv"]).max())
        worst_th, worst_ai = max(worst_th, e_th), max(worst_ai, e_ai)
    assert worst_th <= theta_tol, worst_th
    assert worst_ai <= ainv_tol, worst_ai
    return worst_th, worst_ai
