"""The seeded generator: determinism, length distributions, page dealing and
poison placement."""
import numpy as np
import pytest
import torch

from paper_2504_14489_amd import workloads as W


def test_same_seed_same_bytes_other_seed_other_bytes():
    cfg = W.CONFIGS["tiny"]
    a, b, c = W.make_workload(cfg), W.make_workload(cfg), W.make_workload(cfg, seed=1)
    for name in ("k_pool", "v_pool", "q_pre", "q_dec", "dec_bt", "pre_bt", "dec_lens"):
        assert np.array_equal(getattr(a, name), getattr(b, name))
    assert not np.array_equal(a.k_pool, c.k_pool)


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 7
    x[:4] = [1.00390625, 1.005859375, -3.0e38, 1e-40]   # ties and extremes
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().astype(np.uint16)
    assert np.array_equal(W.f32_to_bf16_bits(x), want)
    assert np.array_equal(W.bf16_bits_to_f32(want), torch.from_numpy(want.view(np.int16)).view(
        torch.bfloat16).float().numpy())


@pytest.mark.parametrize("name", ["tiny", "llama8b", "llama70b", "llama70b_tp8", "longctx8b", "sweep8b"])
def test_decode_lengths_follow_the_config(name):
    cfg = W.CONFIGS[name]
    L = W.draw_decode_lengths(cfg, np.random.Generator(np.random.PCG64(0)))
    assert len(L) == cfg.dec_batch
    assert L.min() >= cfg.dec_len_lo and L.max() <= cfg.dec_len_hi
    if cfg.dec_len_dist == "lognormal":
        assert 1500 < np.median(L) < 2700


def _check_layout(wl: W.Workload):
    S = wl.cfg.page_size
    P = wl.num_pages
    pre_pages = -(-wl.pre_len // S)
    owned = list(wl.pre_bt[:pre_pages])
    for b, L in enumerate(wl.dec_lens):
        np_b = -(-int(L) // S)
        owned += list(wl.dec_bt[b, :np_b])
        assert np.all(wl.dec_bt[b, np_b:] == wl.nan_page)
    assert len(set(owned)) == len(owned), "a page was dealt twice"
    assert all(0 <= p < P - 1 for p in owned)
    unused = np.setdiff1d(np.arange(P), owned)
    assert wl.nan_page in unused
    assert np.all(wl.k_pool[unused] == W.BF16_NAN) and np.all(wl.v_pool[unused] == W.BF16_NAN)
    for bt, L in [(wl.pre_bt, wl.pre_len)] + list(zip(wl.dec_bt, wl.dec_lens)):
        L = int(L)
        if L % S:
            last = bt[L // S]
            assert np.all(wl.k_pool[last, :, L % S:] == W.BF16_SLACK_POISON)
            assert np.all(np.isfinite(W.bf16_bits_to_f32(wl.k_pool[last, :, :L % S])))
        k, v = wl.logical_kv(bt, L)
        assert np.all(np.isfinite(W.bf16_bits_to_f32(k))) and np.all(np.isfinite(W.bf16_bits_to_f32(v)))
    return owned


def test_tiny_layout_and_poison():
    wl = W.make_workload(W.CONFIGS["tiny"])
    assert wl.num_pages == 257 and wl.pre_len == 256
    _check_layout(wl)


def test_sized_to_fit_pool_is_exact():
    cfg = W.custom_config(hq=4, hkv=2, pre_chunks=((5, 11), (16, 7)), dec_batch=7,
                          dec_len_lo=1, dec_len_hi=100, seed=3)
    wl = W.make_workload(cfg)
    owned = _check_layout(wl)
    assert wl.num_pages == len(owned) + 1        # every data page is used, plus the NaN page
    assert np.array_equal(np.sort(wl.perm), np.arange(wl.num_pages - 1))


def test_new_token_kv_views():
    cfg = W.custom_config(hq=4, hkv=2, pre_chunks=((9, 20),), dec_batch=3, dec_len_lo=2,
                          dec_len_hi=50, seed=4)
    wl = W.make_workload(cfg)
    k, v = wl.pre_new_kv(9, 20)
    kk, vv = wl.logical_kv(wl.pre_bt, 29)
    assert np.array_equal(k, kk[9:]) and np.array_equal(v, vv[9:])
    kd, vd = wl.dec_new_kv()
    for b, L in enumerate(wl.dec_lens):
        kk, vv = wl.logical_kv(wl.dec_bt[b], int(L))
        assert np.array_equal(kd[b], kk[-1]) and np.array_equal(vd[b], vv[-1])
