"""Contention-tolerant estimator (paper Sec. 3.3, 3.4): the oracle pinned to
closed forms, then the library's host-side implementation against it."""
import math

import numpy as np
import pytest

from oracle import estimator as E
from paper_2504_14489_amd import mw


# ---------------------------------------------------------------- oracle pins
def test_oracle_recovers_known_coefficients_exactly():
    rng = np.random.default_rng(1)
    th = np.array([3e-7, 1.5e-7, 2e-3, 0.05])
    X, t = [], []
    for _ in range(40):
        bs = int(rng.integers(1, 4))
        n = rng.integers(1, 8192, bs); r = rng.integers(0, 32768, bs)
        X.append(E.prefill_features(n, r))
        # Eq. (1) written out independently of prefill_features
        t.append(th[0] * sum(int(a) ** 2 for a in n) + th[1] * sum(int(a) * int(b) for a, b in zip(n, r))
                 + th[2] * int(n.sum()) + th[3])
    np.testing.assert_allclose(E.fit_relative(np.array(X), np.array(t)), th, rtol=1e-9)
    thd = np.array([2e-6, 4e-3, 0.03])
    X, t = [], []
    for _ in range(30):
        L = rng.integers(1, 20000, int(rng.integers(1, 64)))
        X.append(E.decode_features(L))
        t.append(thd[0] * int((L - 1).sum()) + thd[1] * len(L) + thd[2])  # Eq. (2), r = L - 1
    np.testing.assert_allclose(E.fit_relative(np.array(X), np.array(t)), thd, rtol=1e-9)


def test_oracle_relative_weighting_closed_form():
    # one constant term: argmin sum ((c - t)/t)^2 is sum(1/t) / sum(1/t^2), not mean(t)
    t = np.array([1.0, 2.0, 4.0, 10.0])
    c = E.fit_relative(np.ones((4, 1)), t)[0]
    assert c == pytest.approx(np.sum(1 / t) / np.sum(1 / t ** 2), rel=1e-12)
    assert abs(c - t.mean()) > 1.0


def test_oracle_guard_cells_and_layers():
    assert [E.cell(x, 4) for x in (0, 1, 2, 4, 5, 4096, 4097, 131072)] == [0, 0, 1, 1, 2, 6, 7, 9]
    assert [E.cell(x, 2) for x in (1, 2, 3, 32, 33)] == [0, 1, 2, 5, 6]
    cells = E.guard_build([((4096, 0, 32, 65536, 64), 1.10), ((3000, 0, 17, 50000, 64), 1.25),
                           ((4096, 0, 32, 65536, 128), 1.05)])
    assert E.guard_lookup(cells, (2049, 0, 20, 40000, 64)) == 1.25   # same cell: the maximum
    assert E.guard_lookup(cells, (16, 16, 1, 1, 64)) == 1.25         # empty cell: partition max
    assert E.guard_lookup(cells, (16, 16, 1, 1, 32)) == 1.25         # unknown partition: global max
    assert E.guard_lookup({}, (1, 1, 1, 1, 64)) == 1.0
    # Sec. 3.4: T_d = 30 ms next to a 1000 ms prefill of an 80-layer model -> 3 layers
    assert E.prefill_layers(30.0, 1000.0, 80) == 3
    assert E.prefill_layers(5000.0, 10.0, 32) == 32 and E.prefill_layers(1e-6, 10.0, 32) == 1


# ---------------------------------------------------- library against oracle
def _noisy_samples(rng, n_samples):
    th = np.array([4e-7, 2e-7, 1e-3, 0.02])
    out = []
    for _ in range(n_samples):
        bs = int(rng.integers(1, 4))
        n = rng.integers(1, 4096, bs); r = rng.integers(0, 16384, bs)
        t = float(E.prefill_features(n, r) @ th) * float(rng.uniform(0.9, 1.1))
        out.append((n, r, t))
    return out


def test_predictor_fit_and_predictions_match_oracle():
    rng = np.random.default_rng(7)
    p = mw.mw_predictor_create()
    try:
        per_cus = {}
        for cus in (64, 128):
            smp = _noisy_samples(rng, 25)
            per_cus[cus] = smp
            for n, r, t in smp:
                mw.mw_predictor_add_prefill(p, cus, n, r, t)
        dsmp = []
        for _ in range(20):
            L = rng.integers(1, 9000, int(rng.integers(1, 48)))
            t = (1e-5 * (L - 1).sum() + 2e-3 * len(L) + 0.01) * float(rng.uniform(0.92, 1.08))
            dsmp.append((L, t))
            mw.mw_predictor_add_decode(p, 192, L, t)
        mw.mw_predictor_fit(p)
        for cus, smp in per_cus.items():
            X = np.array([E.prefill_features(n, r) for n, r, _ in smp]); t = np.array([s[2] for s in smp])
            ref = E.fit_relative(X, t)
            np.testing.assert_allclose(mw.mw_predictor_coefficients(p, 0, cus), ref, rtol=1e-8)
            for n, r, _ in smp[:5]:
                assert mw.mw_predictor_prefill_ms(p, cus, n, r) == pytest.approx(
                    float(E.prefill_features(n, r) @ ref), rel=1e-9)
        X = np.array([E.decode_features(L) for L, _ in dsmp]); t = np.array([s[1] for s in dsmp])
        ref = E.fit_relative(X, t)
        np.testing.assert_allclose(mw.mw_predictor_coefficients(p, 1, 192)[:3], ref, rtol=1e-8)
        L = dsmp[0][0]
        assert mw.mw_predictor_decode_ms(p, 192, L) == pytest.approx(float(E.decode_features(L) @ ref),
                                                                      rel=1e-9)
    finally:
        mw.mw_predictor_destroy(p)


def test_predictor_unexercised_term_and_errors():
    p = mw.mw_predictor_create()
    try:
        with pytest.raises(mw.MWError) as ei:
            mw.mw_predictor_fit(p)
        assert ei.value.status == mw.MW_ERR_NOT_READY
        rng = np.random.default_rng(3)
        X, t = [], []
        for _ in range(10):  # no reused tokens at all: the n*r term stays 0
            n = rng.integers(1, 2048, 2)
            tt = float(1e-6 * (n ** 2).sum() + 1e-3 * n.sum() + 0.05)
            mw.mw_predictor_add_prefill(p, 32, n, [0, 0], tt)
            X.append(E.prefill_features(n, [0, 0])); t.append(tt)
        mw.mw_predictor_fit(p)
        th = mw.mw_predictor_coefficients(p, 0, 32)
        assert th[1] == 0.0
        np.testing.assert_allclose(th, E.fit_relative(np.array(X), np.array(t)), rtol=1e-8, atol=1e-18)
        with pytest.raises(mw.MWError) as ei:
            mw.mw_predictor_prefill_ms(p, 64, [10], [0])   # no model for 64 CUs
        assert ei.value.status == mw.MW_ERR_NOT_READY
        for bad in (lambda: mw.mw_predictor_add_prefill(p, 32, [0], [0], 1.0),
                    lambda: mw.mw_predictor_add_prefill(p, 32, [5], [-1], 1.0),
                    lambda: mw.mw_predictor_add_prefill(p, 32, [5], [0], -1.0),
                    lambda: mw.mw_predictor_add_prefill(p, 32, [5], [0], float("nan")),
                    lambda: mw.mw_predictor_add_decode(p, 0, [5], 1.0),
                    lambda: mw.mw_predictor_add_decode(p, 32, [0], 1.0)):
            with pytest.raises(mw.MWError) as ei:
                bad()
            assert ei.value.status == mw.MW_ERR_INVALID_ARG
    finally:
        mw.mw_predictor_destroy(p)


def test_guard_matches_oracle():
    rng = np.random.default_rng(11)
    g = mw.mw_guard_create()
    try:
        samples = []
        for _ in range(300):
            key = (int(rng.choice([512, 2048, 8192, 30000])), int(rng.choice([0, 1024, 16384])),
                   int(rng.integers(1, 200)), int(rng.integers(0, 2_000_000)), int(rng.choice([64, 128, 192])))
            s = float(rng.uniform(0.98, 1.3))
            samples.append((key, s))
            mw.mw_guard_add(g, *key, s)
        cells = E.guard_build(samples)
        for _ in range(500):
            key = (int(rng.integers(0, 40000)), int(rng.integers(0, 40000)), int(rng.integers(1, 300)),
                   int(rng.integers(0, 3_000_000)), int(rng.choice([32, 64, 128, 192])))
            assert mw.mw_guard_lookup(g, *key) == E.guard_lookup(cells, key)
        with pytest.raises(mw.MWError):
            mw.mw_guard_add(g, 1, 1, 0, 1, 64, 1.1)
        with pytest.raises(mw.MWError):
            mw.mw_guard_add(g, 1, 1, 1, 1, 64, 0.0)
    finally:
        mw.mw_guard_destroy(g)
    g = mw.mw_guard_create()
    try:
        assert mw.mw_guard_lookup(g, 1, 1, 1, 1, 64) == 1.0
    finally:
        mw.mw_guard_destroy(g)


def test_prefill_layers_matches_oracle():
    rng = np.random.default_rng(5)
    for _ in range(200):
        td, tp, nl = float(rng.uniform(0.01, 50)), float(rng.uniform(0.05, 5000)), int(rng.integers(1, 128))
        assert mw.mw_prefill_layers(td, tp, nl) == E.prefill_layers(td, tp, nl)
    for bad in ((0.0, 1.0, 32), (1.0, 0.0, 32), (1.0, 1.0, 0), (math.inf, 1.0, 32)):
        with pytest.raises(mw.MWError):
            mw.mw_prefill_layers(*bad)


def test_engine_estimate_from_a_profile(tmp_path):
    """The engine's estimator reads a profiling run: the solo predictions
    reproduce times generated from Eqs. (1)-(2), and the guard returns the
    measured slowdown of the matching cell."""
    import json
    from paper_2504_14489_amd.engine import Estimate
    th_p = (2e-8, 1e-8, 3e-5, 0.01)   # ms per n^2, n*r, n, constant
    th_d = (1e-5, 2e-4, 0.02)         # ms per reused token, per sequence, constant

    def t_pre(n, r):
        return th_p[0] * n * n + th_p[1] * n * r + th_p[2] * n + th_p[3]

    def t_dec(lens):
        return th_d[0] * sum(L - 1 for L in lens) + th_d[1] * len(lens) + th_d[2]

    prof = {"model": {"num_q_heads": 32, "num_kv_heads": 8, "head_dim": 128, "page_size": 16},
            "prefill": [], "decode": [], "pairs": []}
    for n in (1024, 4096, 16384):
        for r in (0, 4096, 16384):
            prof["prefill"].append({"cus": 64, "n": n, "r": r, "ms": t_pre(n, r), "grid": True})
    for bs in (8, 32, 128):
        for L in (1024, 4096, 16384):
            prof["decode"].append({"cus": 192, "lens": [L] * bs, "ms": t_dec([L] * bs), "grid": True})
    prof["pairs"].append({"prefill_cus": 64, "prefill_new": 2048, "prefill_reused": 0, "decode_batch": 64,
                          "decode_reused": 64 * 2047, "slowdown": 1.17})
    path = tmp_path / "profile.json"
    path.write_text(json.dumps(prof))
    est = Estimate(str(path))
    try:
        lens = [2048] * 64
        sp, sd, slow = est.layers(64, [2048], [0], lens)
        assert sp == pytest.approx(t_pre(2048, 0), rel=1e-6)
        assert sd == pytest.approx(t_dec(lens), rel=1e-6)
        assert slow == pytest.approx(1.17)
    finally:
        est.close()


# ------------------------------- launch-imbalance factor (not from the paper)
def test_oracle_launch_imbalance_hand_cases():
    # 64 new tokens, 1 kv head of 1 query head, 2 CUs: the one 64-position pair
    # is fewer than the CUs -> 32-position blocks, two work-groups per CU; the two
    # blocks (1 key tile each) land on different CUs, each alone: factor 1 / 0.9
    path, k = E.prefill_launch([64], [0], 1, 1, 2)
    assert path == 1 and k == pytest.approx(1 / 0.9, rel=1e-12)
    # 128 tokens on 1 CU: 64-position blocks 1 and 0 paired in one work-group
    # (2 + 1 tiles): nothing to balance
    path, k = E.prefill_launch([128], [0], 1, 1, 1)
    assert path == 0 and k == pytest.approx(1.0, rel=1e-12)
    # 192 tokens on 2 CUs: pairs (2, 0) with 3 + 1 tiles and (1) alone with 2:
    # CU loads 4 and 2 against 3 each if even -> 4 * 2 / 6
    path, k = E.prefill_launch([192], [0], 1, 1, 2)
    assert path == 0 and k == pytest.approx(4 / 3, rel=1e-12)
    # one 32-position block over 4064 cached tokens (64 tiles) on 4 CUs: cut in 8
    # pieces of 8 tiles, two per CU -> even
    path, k = E.prefill_launch([32], [4064], 1, 1, 4)
    assert path == 1 and k == pytest.approx(1.0, rel=1e-12)
    # 8 kv heads of 4 query heads, 4096 tokens on 64 CUs: 32 pairs x 8 heads = 256
    # equal pairs fill 4 whole rounds -> even
    path, k = E.prefill_launch([4096], [0], 8, 4, 64)
    assert path == 0 and k == pytest.approx(1.0, rel=1e-12)


def test_oracle_launch_dispatch_window():
    # 141 tokens over 3000 cached, 2 kv heads, 3 CUs: 4 pairs do not fill 2 whole
    # rounds of 3 -> single 64-position blocks 2, 2, 1, 1, 0, 0 (heads fastest) of
    # 50, 50, 49, 49, 48, 48 tiles; window 0.05 * 294 / 6.  Work-groups 0-2 take
    # CUs 0-2 (free at 50, 50, 49); work-group 3 sees all three inside the window,
    # equal counts -> CU 0; then CU 1, CU 2: loads 99, 98, 97 (the earliest-free
    # rule alone would give 98 each)
    path, k = E.prefill_launch([141], [3000], 2, 1, 3)
    assert path == 0 and k == pytest.approx(99 * 3 / 294, rel=1e-12)
    # 130 tokens over 576 cached, 1 kv head, 6 CUs: 32-position blocks cut into
    # pieces, 15 work-groups of 4,4,4,3,4,4 | 3,4,4,3,3,4 | 3,3,4 tiles (54 in all)
    # on 12 slots.  The first 12 fill slot 0 then slot 1 of CUs 0-5; at time 3 the
    # free slots are slot 0 of CU 3 and slot 1 of CUs 0, 3, 4, every CU holding 2:
    # CU 3, then CU 0 (2 < 3), then CU 4 (2 < 3) -> loads 10, 8, 8, 9, 11, 8 and
    # 11 * 6 / 54 (the lower-slot rule alone gives CU 3 both tail work-groups: 13)
    path, k = E.prefill_launch([130], [576], 1, 1, 6)
    assert path == 1 and k == pytest.approx(11 * 6 / 54, rel=1e-12)


def test_oracle_launch_imbalance_at_least_one():
    rng = np.random.default_rng(5)
    for _ in range(60):
        bs = int(rng.integers(1, 4))
        n = rng.integers(1, 2500, bs); r = rng.integers(0, 9000, bs)
        cus = int(rng.choice([8, 32, 96, 256]))
        _, k = E.prefill_launch(n, r, int(rng.choice([1, 2, 8])), int(rng.choice([1, 4, 8])), cus)
        assert k >= 1.0 - 1e-12


def _launch_samples(rng, hkv, group, cus, count):
    th = {0: np.array([4e-8, 2e-8, 1e-5, 0.01]), 2: np.array([6e-8, 3e-8, 2e-5, 0.015])}
    out = []
    for i in range(count):
        bs = int(rng.integers(1, 3))
        n = rng.integers(1, 300 if i % 2 else 3000, bs); r = rng.integers(0, 20000, bs)
        ph, x = E.prefill_features_launch(n, r, hkv, group, cus)
        out.append((ph, n, r, x, float(x @ th[ph]) * float(rng.uniform(0.95, 1.05))))
    return out


def test_predictor_launch_shape_matches_oracle():
    rng = np.random.default_rng(11)
    hq, hkv = 32, 8
    p = mw.mw_predictor_create()
    try:
        mw.mw_predictor_add_decode(p, 64, [100, 200], 0.02)  # decode samples may come first
        mw.mw_predictor_set_launch_shape(p, hq, hkv)
        samples = {}
        for cus in (32, 128):
            for ph, n, r, x, t in _launch_samples(rng, hkv, hq // hkv, cus, 40):
                samples.setdefault((ph, cus), []).append((n, r, x, t))
                mw.mw_predictor_add_prefill(p, cus, n, r, t)
        mw.mw_predictor_fit(p)
        assert {k[0] for k in samples} == {0, 2}
        for (ph, cus), smp in samples.items():
            assert len(smp) >= 4
            ref = E.fit_relative(np.array([s[2] for s in smp]), np.array([s[3] for s in smp]))
            np.testing.assert_allclose(mw.mw_predictor_coefficients(p, ph, cus), ref, rtol=1e-7)
            for n, r, x, _ in smp[:4]:
                assert mw.mw_predictor_prefill_ms(p, cus, n, r) == pytest.approx(float(x @ ref), rel=1e-9)
    finally:
        mw.mw_predictor_destroy(p)


def test_predictor_launch_shape_long_prefixes_match_oracle():
    # split launches over long prefixes, where many work-groups tie
    rng = np.random.default_rng(17)
    p = mw.mw_predictor_create()
    try:
        mw.mw_predictor_set_launch_shape(p, 32, 8)
        th = np.array([5e-8, 2e-8, 3e-5, 0.02])
        smp = []
        for _ in range(12):
            n = [int(rng.integers(100, 1500))]; r = [int(rng.integers(0, 60000))]
            ph, x = E.prefill_features_launch(n, r, 8, 4, 96)
            assert ph == 2
            t = float(x @ th) * float(rng.uniform(0.95, 1.05))
            smp.append((n, r, x, t))
            mw.mw_predictor_add_prefill(p, 96, n, r, t)
        mw.mw_predictor_fit(p)
        ref = E.fit_relative(np.array([s[2] for s in smp]), np.array([s[3] for s in smp]))
        np.testing.assert_allclose(mw.mw_predictor_coefficients(p, 2, 96), ref, rtol=1e-7)
        for n, r, x, _ in smp:
            assert mw.mw_predictor_prefill_ms(p, 96, n, r) == pytest.approx(float(x @ ref), rel=1e-9)
    finally:
        mw.mw_predictor_destroy(p)


def test_predictor_launch_shape_rules_and_fallback():
    p = mw.mw_predictor_create()
    try:
        with pytest.raises(mw.MWError):
            mw.mw_predictor_set_launch_shape(p, 30, 8)  # not a multiple of the kv heads
        mw.mw_predictor_set_launch_shape(p, 32, 8)
        rng = np.random.default_rng(2)
        smp = []
        for _ in range(8):  # long chunks only: every sample on the 8-wave path
            n = [int(rng.integers(6000, 9000))]; r = [int(rng.integers(0, 4000))]
            ph, x = E.prefill_features_launch(n, r, 8, 4, 64)
            assert ph == 0
            t = float(x @ np.array([3e-8, 1e-8, 2e-5, 0.02]))
            smp.append((x, t))
            mw.mw_predictor_add_prefill(p, 64, n, r, t)
        with pytest.raises(mw.MWError):
            mw.mw_predictor_set_launch_shape(p, 32, 8)  # prefill samples already added
        mw.mw_predictor_fit(p)
        ref = E.fit_relative(np.array([s[0] for s in smp]), np.array([s[1] for s in smp]))
        # a short chunk takes the 4-wave path, which has no model: the 8-wave
        # path's model is used with the short chunk's own (scaled) terms
        ph, x = E.prefill_features_launch([100], [500], 8, 4, 64)
        assert ph == 2
        assert mw.mw_predictor_prefill_ms(p, 64, [100], [500]) == pytest.approx(float(x @ ref), rel=1e-9)
        with pytest.raises(mw.MWError) as ei:
            mw.mw_predictor_coefficients(p, 2, 64)
        assert ei.value.status == mw.MW_ERR_NOT_READY
    finally:
        mw.mw_predictor_destroy(p)
