"""The estimator's offline profiling on the GPU (a small grid): solo runs and
multiplexed pairs on a CU partition, the predictor fitted through the C ABI
and the contention guard filled."""
import json

import pytest

from tests.helpers import say

pytestmark = pytest.mark.gpu


def test_profiling_quick_sweep(tmp_path):
    say("estimator profiling, quick grid on 64/192")
    out = tmp_path / "est.json"
    from paper_2504_14489_amd import profiling
    profiling.main(["--quick", "--prefill-cus", "64", "--held-out", "4", "--reps", "3", "--out", str(out)])
    d = json.loads(out.read_text())
    assert len(d["prefill"]) == 6 + 4 and len(d["decode"]) == 4 + 4 and len(d["pairs"]) == 24
    assert all(s["ms"] > 0 for s in d["prefill"] + d["decode"])
    # prefill: the 8-wave path's and the 4-wave path's coefficients (zeros for
    # a path without a model: the quick grid's chunks are mostly short)
    th = d["predictor"]["prefill"]["64"]["theta"]
    assert len(th) == 8 and all(map(lambda v: v == v, th)) and any(v != 0 for v in th)
    assert "192" in d["predictor"]["decode"]
    assert d["guard"]["pairs_measured"] >= 1 and d["guard"]["max_slowdown"] > 0.5
