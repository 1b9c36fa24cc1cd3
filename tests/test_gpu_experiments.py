"""The quality-experiment runner on the GPU (synthetic analogs of Sec. 5):
it produces every table, and the learned policy shows the paper's
qualitative results on the simulator: lower energy and EDP than the top
clock after convergence, and a learned clock near the offline optimum."""
import math

import pytest

from gpu_helpers import say
from paper_2508_01744_amd import experiments as E

pytestmark = pytest.mark.gpu


def test_report_small_run():
    rep = E.report("cfg2pe", B=256, T=600)
    say(E.markdown(rep))
    post = rep["vs_default"]["post"]
    assert post["energy"]["diff"] < -10.0
    assert post["edp"]["diff"] < 0.0
    assert rep["switched_fraction"] > 0.5
    assert len(rep["frequency"]) == 5
    for row in rep["frequency"]:
        assert row["abs_deviation"] < 25.0, row
    assert set(rep["ablation"]) == {"full", "no-grain", "no pruning"}
    for row in rep["ablation"].values():
        assert all(math.isfinite(row[m]["mean"]) and row[m]["cv"] >= 0.0 for m in E.METRICS)
    assert len(rep["rolling_reward"]) >= 5
