"""Loader of the hand-worked LinUCB example in tests/golden/."""
import os
from fractions import Fraction

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _fracs(s):
    return [Fraction(v) for v in s.split(",")]


def load_worked_example(path=os.path.join(GOLDEN, "linucb_worked_example.txt")):
    ex = dict(steps=[], final_Ainv={}, final_theta={})
    with open(path) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("lambda") or line.startswith("alpha"):
                key, val = [p.strip() for p in line.split("=")]
                ex[key] = Fraction(val)
            elif line.startswith("step "):
                fields = dict(p.split("=") for p in line[5:].split())
                ex["steps"].append(dict(x=_fracs(fields["x"]), mean=_fracs(fields["mean"]),
                                        quad=_fracs(fields["quad"]),
                                        action=int(fields["action"]),
                                        reward=Fraction(fields["reward"])))
            elif line.startswith("final_Ainv") or line.startswith("final_theta"):
                kind, arm, val = line.split()
                k = int(arm.split("=")[1])
                if kind == "final_Ainv":
                    ex[kind][k] = [_fracs(row) for row in val.split(";")]
                else:
                    ex[kind][k] = _fracs(val)
    K = len(ex["final_theta"])
    ex["final_Ainv"] = [ex["final_Ainv"][k] for k in range(K)]
    ex["final_theta"] = [ex["final_theta"][k] for k in range(K)]
    return ex


def load_page_hinkley_example(path=os.path.join(GOLDEN, "page_hinkley_worked_example.txt")):
    """The hand-worked Page-Hinkley example: parameters (delta, lambda, window,
    min_rounds) and, per round, the reward entering it, the state after it
    (n, mean, up, up_min, dn, dn_min), the margin, the alarm flag and the mode."""
    ex = dict(rounds=[])
    with open(path) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("round "):
                f = dict(p.split("=") for p in line[6:].split())
                ex["rounds"].append(dict(
                    t=int(f["t"]), r=Fraction(f["r"]), alarm=int(f["alarm"]), mode=int(f["mode"]),
                    state=[Fraction(f[k]) for k in ("n", "mean", "up", "up_min", "dn", "dn_min")],
                    margin=Fraction(f["margin"])))
            else:
                key, val = [p.strip() for p in line.split("=")]
                ex[key] = Fraction(val) if key in ("delta", "lambda") else int(val)
    return ex
