"""The fp64 oracle against the mathematics it follows (CPU only)."""
import pytest

import oracle_pins as pins
from oracle import load_library


@pytest.fixture(scope="module")
def lib():
    return load_library()


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(lib, pin):
    pin(lib)


def test_worked_example_is_self_consistent():
    """The hand derivation's numbers agree with Eq. 1/3/4/5 redone in exact
    rationals with the 2x2 adjugate inverse (catches typos in the fixture)."""
    from fractions import Fraction as F
    from golden_example import load_worked_example
    ex = load_worked_example()
    lam = ex["lambda"]
    A = [[[lam, F(0)], [F(0), lam]] for _ in range(2)]
    b = [[F(0), F(0)] for _ in range(2)]

    def inv(M):
        det = M[0][0] * M[1][1] - M[0][1] * M[1][0]
        return [[M[1][1] / det, -M[0][1] / det], [-M[1][0] / det, M[0][0] / det]]

    for step in ex["steps"]:
        x = step["x"]
        for k in range(2):
            Ai = inv(A[k])
            theta = [Ai[0][0] * b[k][0] + Ai[0][1] * b[k][1], Ai[1][0] * b[k][0] + Ai[1][1] * b[k][1]]
            mean = theta[0] * x[0] + theta[1] * x[1]
            quad = sum(x[p] * Ai[p][q] * x[q] for p in range(2) for q in range(2))
            assert mean == step["mean"][k] and quad == step["quad"][k]
        a = step["action"]
        for p in range(2):
            for q in range(2):
                A[a][p][q] += x[p] * x[q]
            b[a][p] += step["reward"] * x[p]
    for k in range(2):
        Ai = inv(A[k])
        assert Ai == ex["final_Ainv"][k]
        theta = [Ai[0][0] * b[k][0] + Ai[0][1] * b[k][1], Ai[1][0] * b[k][0] + Ai[1][1] * b[k][1]]
        assert theta == ex["final_theta"][k]


def test_page_hinkley_example_is_self_consistent():
    """The hand derivation's numbers agree with the test's definition redone
    in exact rationals: each running mean recomputed from the rewards since
    the last restart, the cumulative sums and their minima rebuilt from them
    (catches typos in the fixture)."""
    from fractions import Fraction as F
    from golden_example import load_page_hinkley_example
    ex = load_page_hinkley_example()
    delta, lam = ex["delta"], ex["lambda"]
    seg, last, mode = [], 0, -1
    for rd in ex["rounds"]:
        t = rd["t"]
        if mode < 0:
            seg.append(rd["r"])
            sums = [F(0), F(0)]
            mins = [F(0), F(0)]
            for q in range(len(seg)):
                rbar = sum(seg[:q + 1]) / (q + 1)
                sums = [sums[0] + seg[q] - rbar - delta, sums[1] + rbar - seg[q] - delta]
                mins = [min(mins[0], sums[0]), min(mins[1], sums[1])]
            stat = max(sums[0] - mins[0], sums[1] - mins[1])
            margin = lam - stat
            alarm = int(stat > lam)
            state = [F(len(seg)), sum(seg) / len(seg), sums[0], mins[0], sums[1], mins[1]]
            if alarm:
                last, seg, state = t, [], [F(0)] * 6
            if t >= ex["min_rounds"] and t - last >= ex["window"]:
                mode = t
        else:
            alarm = 0
        assert rd["alarm"] == alarm and rd["mode"] == mode and rd["margin"] == margin, t
        assert rd["state"] == state, (t, rd["state"], state)
