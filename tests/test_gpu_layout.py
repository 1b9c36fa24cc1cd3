"""Both record layouts on the GPU against the oracle: packed tails (with
pruning on, as here: an exploring instance streams more than 16 KB of
records per step) and tails padded to whole chunks (16 KB or less), at every
supported d, with an arm count that leaves the last block of records
part-filled.

Open loop (the same contexts and rewards to both sides); afterwards the
final models are compared through the export kernel, and the raw records
are checked for what the layout promises: zero padding floats with padded
tails, and zero slots past K in the last block."""
import numpy as np
import pytest
import torch

import parity
from gpu_helpers import compare_model, random_contexts, run_open_loop, say
from paper_2508_01744_amd import _lib as L

pytestmark = pytest.mark.gpu


def _decode(arms, K, d, tf):
    """theta [B][K][d] and the upper-triangular factor S [B][K][d][d] from the
    raw records [B][blocks][NB*chunks][4], following the layout that
    include/agft.h documents for agft_state_view.arms."""
    B = arms.shape[0]
    G, nb = d // 2, 64 // d
    M, T = G * (d // 4), G * tf // 4
    theta = np.zeros((B, K, d), np.float32)
    S = np.zeros((B, K, d, d), np.float32)
    for k in range(K):
        blk, r = arms[:, k // nb], k % nb
        main = blk[:, r * M:(r + 1) * M]                          # [B][M][4]
        tail = blk[:, nb * M + r * T:nb * M + (r + 1) * T].reshape(B, -1)
        for j in range(G):
            for e in range(d + 3):
                v = main[:, (e // 4) * G + j, e % 4] if e < d else tail[:, tf * j + e - d]
                if e <= j:
                    S[:, k, e, j] = v
                elif e <= d:
                    S[:, k, d - e, d - 1 - j] = v
                else:
                    theta[:, k, 2 * j + e - d - 1] = v
    return theta, S

# (d, K, expected tail floats): K*4*(d + d(d+1)/2) bytes against 16 KB, and
# K % (64/d) != 0 in every case
CASES = [(8, 21, 4), (8, 100, 3), (16, 10, 4), (16, 30, 3), (32, 5, 4), (32, 9, 3)]


@pytest.mark.parametrize("d,K,tf", CASES)
def test_layout_open_loop(d, K, tf):
    assert (K * 4 * (d + d * (d + 1) // 2) > 16384) == (tf == 3)
    cfg = dict(B=9, K=K, d=d, lam=1.0, alpha0=0.5, sched=0, prune=1, period=13, heuristics=None)
    T = 70
    X, R = random_contexts(1000 + 10 * d + K, T, cfg["B"], d)
    say(f"[layout] d={d} K={K} tf={tf} T={T}")
    a, m, s, tuner, _ = run_open_loop(cfg, X, R)
    st = parity.compare_open_loop(f"layout d={d} K={K}", cfg, X, R, a, m, s)
    compare_model(tuner, st["oracle"], range(cfg["B"]), 1e-3, 1e-4)

    code, v = L.agft_get_state(tuner.h)
    L.check("agft_get_state", code)
    nb, G = 64 // d, d // 2
    assert v.tail_floats == tf and v.block_arms == nb
    assert v.chunks == G * (d // 4) + G * tf // 4
    C, MAIN, TAIL = v.chunks, G * (d // 4), G * tf // 4
    arms = tuner.view()["arms"].cpu().numpy()          # [B][blocks][NB*C][4]
    assert arms.shape[1] == (K + nb - 1) // nb
    last = arms[:, -1]
    for r in range(K % nb, nb):                        # slots past K in the last block
        assert not last[:, r * MAIN:(r + 1) * MAIN].any()
        assert not last[:, nb * MAIN + r * TAIL:nb * MAIN + (r + 1) * TAIL].any()
    if tf == 4:                                        # float 4j+3 of every tail slice
        tails = arms[:, :, nb * MAIN:, :]
        assert not tails[..., 3].any()
    # the records decoded as the header documents them give the exported model
    theta, S = _decode(arms, K, d, tf)
    th, ai = tuner.export(theta=True, ainv=True)
    assert np.array_equal(theta, th.cpu().numpy())
    ainv = np.einsum("bkij,bklj->bkil", S.astype(np.float64), S.astype(np.float64))
    ref = ai.cpu().numpy().astype(np.float64)
    assert np.abs(ainv - ref).max() <= 1e-5 * max(1.0, np.abs(ref).max())
    say(f"[layout] d={d} K={K}: max score err {st['max_score_err']:.2e}, "
        f"forced {st['forced']}/{st['decisions']}")
    torch.cuda.synchronize()
