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
