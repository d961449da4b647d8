"""Host side of the estimator profiling tool: re-scoring a saved sweep (no GPU)."""
import json

import numpy as np

from paper_2504_14489_amd import profiling


def _fake_sweep():
    rng = np.random.default_rng(9)
    th_p = np.array([4e-8, 2e-8, 1e-5, 0.01])
    th_d = np.array([1e-6, 2e-4, 0.015])
    res = {"model": {"num_q_heads": 32, "num_kv_heads": 8, "head_dim": 128, "page_size": 16},
           "grid": {"prefill_new": [512, 4096], "prefill_reused": [0, 8192], "decode_batch": [1, 64],
                    "decode_len": [1024, 8192], "max_decode_tokens": 1 << 22,
                    "guard": {"prefill_new": [4096], "prefill_reused": [0], "decode_batch": [64],
                              "decode_len": [1024]}},
           "prefill": [], "decode": [], "pairs": [], "seconds": 1.0,
           "command": "python3 -m paper_2504_14489_amd.profiling --out sweep.json"}
    for cus in (64, 192):
        for i in range(30):
            n, r = int(rng.integers(4000, 9000)), int(rng.integers(0, 20000))
            t = float(np.array([n * n, n * r, n, 1.0]) @ th_p) * float(rng.uniform(0.97, 1.03))
            res["prefill"].append({"cus": cus, "n": n, "r": r, "ms": t, "grid": i < 24})
            lens = [int(x) for x in rng.integers(1000, 9000, int(rng.integers(8, 64)))]
            t = float(np.array([sum(lens), len(lens), 1.0]) @ th_d) * float(rng.uniform(0.97, 1.03))
            res["decode"].append({"cus": 256 - cus, "lens": lens, "ms": t, "grid": i < 24})
        res["pairs"].append({"prefill_cus": cus, "prefill_new": 4096, "prefill_reused": 0, "decode_batch": 64,
                             "decode_reused": 64 * 1023, "slowdown": 1.1 + cus / 1000})
    return res


def test_rescore_refits_and_writes_the_table(tmp_path):
    src, out, table = tmp_path / "sweep.json", tmp_path / "scored.json", tmp_path / "table.md"
    src.write_text(json.dumps(_fake_sweep()))
    profiling.main(["--rescore", str(src), "--out", str(out), "--table", str(table)])
    res = json.loads(out.read_text())
    for phase in ("prefill", "decode"):
        assert len(res["predictor"][phase]) == 2
        for e in res["predictor"][phase].values():
            # 3% noise on the samples: the fit's deviations stay near it
            assert e["max_dev"]["train"] < 0.08 and e["max_dev"]["held_out"] < 0.08
            assert e["max_dev"]["held_out_long"] <= e["max_dev"]["held_out"]
    assert abs(res["guard"]["max_slowdown"] - 1.292) < 1e-12 and res["guard"]["pairs_measured"] == 2
    text = table.read_text()
    assert "sweep.json" in text and "--rescore" in text and "calls of 0.1 ms or more" in text
