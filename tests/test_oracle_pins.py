"""Pins of the CPU oracle to results fixed by something other than itself.

* torch's scaled_dot_product_attention (a library routine; float64 on CPU,
  explicit boolean mask, ``enable_gqa`` for the head grouping) on the dense,
  unpaged arrays;
* a numpy float64 brute force in matrix form with an explicit mask matrix;
* closed forms: q = 0 gives the mean of the visible V rows; one visible key
  gives its V row; a constant V gives that constant; two keys give logistic
  weights; the worked example in ``tests/golden/worked_example.json``;
* invariants the definition implies: page-permutation invariance, chunked
  prefill equal to unchunked (Sec. 1: each chunk reads all earlier chunks'
  KV), keys after a row's position never matter (causal), decode over L
  tokens equal to the last prefill row over L tokens (Sec. 3.3, Table
  "tab:theory_cost": decode attends r + 1 keys), grouped-query attention equal
  to multi-head attention with repeated KV heads, thread-count independence,
  softmax weights summing to one, and the split/merge identity.

These tests never touch a GPU.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2504_14489_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def dense_inputs(wl: W.Workload, r: int, n: int):
    """Logical (unpaged) float64 arrays for prefill rows [r, r+n) of the
    prefill sequence: q [n][Hq][D], k/v [r+n][Hkv][D]."""
    k, v = wl.logical_kv(wl.pre_bt, r + n)
    q = W.bf16_bits_to_f32(wl.q_pre[r:r + n]).astype(np.float64)
    return q, W.bf16_bits_to_f32(k).astype(np.float64), W.bf16_bits_to_f32(v).astype(np.float64)


def sdpa_prefill(q, k, v, r, scale):
    """torch SDPA with an explicit bottom-right causal mask over the prefix."""
    n, L = q.shape[0], k.shape[0]
    mask = torch.arange(L)[None, :] <= (r + torch.arange(n))[:, None]
    out = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).permute(1, 0, 2)[None],
        torch.from_numpy(k).permute(1, 0, 2)[None],
        torch.from_numpy(v).permute(1, 0, 2)[None],
        attn_mask=mask, scale=scale, enable_gqa=True)
    return out[0].permute(1, 0, 2).numpy()


def numpy_bruteforce(q, k, v, r, scale):
    """Matrix-form attention with an explicit mask matrix (float64)."""
    n, hq, d = q.shape
    L, hkv, _ = k.shape
    g = hq // hkv
    out = np.zeros((n, hq, d))
    mask = np.arange(L)[None, :] <= (r + np.arange(n))[:, None]
    for h in range(hq):
        S = (q[:, h, :] @ k[:, h // g, :].T) * scale
        S = np.where(mask, S, -np.inf)
        S = S - S.max(axis=1, keepdims=True)
        P = np.exp(S)
        P = P / P.sum(axis=1, keepdims=True)
        out[:, h, :] = P @ v[:, h // g, :]
    return out


SHAPES = [
    # (hq, hkv, d, page, n, r)
    (1, 1, 16, 1, 1, 0),
    (2, 1, 16, 4, 3, 5),
    (4, 2, 16, 16, 17, 0),
    (4, 2, 128, 16, 17, 33),
    (8, 2, 128, 16, 3, 16),
    (8, 8, 16, 4, 17, 5),
    (8, 1, 128, 16, 1, 33),
    (4, 4, 128, 1, 17, 16),
]


@pytest.mark.parametrize("hq,hkv,d,page,n,r", SHAPES)
def test_oracle_matches_library_sdpa_and_bruteforce(hq, hkv, d, page, n, r):
    cfg = W.custom_config(hq=hq, hkv=hkv, head_dim=d, page_size=page,
                          pre_chunks=((r, n),), dec_batch=2, dec_len_lo=1, dec_len_hi=9,
                          seed=hq * 1000 + n * 10 + r)
    wl = W.make_workload(cfg, q_scale=3.0)
    scale = 1.0 / math.sqrt(d)
    got = oracle.prefill(wl.q_pre[r:r + n], wl.k_pool, wl.v_pool, wl.pre_bt, r, scale=scale)
    q, k, v = dense_inputs(wl, r, n)
    ref = sdpa_prefill(q, k, v, r, scale)
    bf = numpy_bruteforce(q, k, v, r, scale)
    assert np.all(np.isfinite(got))
    assert np.max(np.abs(got - ref)) <= 1e-12
    assert np.max(np.abs(got - bf)) <= 1e-12


def test_decode_matches_library_sdpa():
    cfg = W.custom_config(hq=8, hkv=2, pre_chunks=((0, 4),), dec_batch=5,
                          dec_len_lo=1, dec_len_hi=70, seed=7)
    wl = W.make_workload(cfg)
    scale = 1.0 / math.sqrt(128)
    got = oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens, scale=scale)
    for b, L in enumerate(wl.dec_lens):
        k, v = wl.logical_kv(wl.dec_bt[b], int(L))
        q = W.bf16_bits_to_f32(wl.q_dec[b:b + 1]).astype(np.float64)
        ref = sdpa_prefill(q, W.bf16_bits_to_f32(k).astype(np.float64),
                           W.bf16_bits_to_f32(v).astype(np.float64), int(L) - 1, scale)
        assert np.max(np.abs(got[b] - ref[0])) <= 1e-12


def _tiny_pool(hq, hkv, d, page, length, seed=0):
    cfg = W.custom_config(hq=hq, hkv=hkv, head_dim=d, page_size=page,
                          pre_chunks=((0, length),), dec_batch=0, seed=seed)
    return W.make_workload(cfg)


def test_zero_query_gives_mean_of_visible_values():
    wl = _tiny_pool(4, 2, 128, 16, 40)
    q = np.zeros((5, 4, 128), dtype=np.uint16)          # +0.0 in bf16
    r = 35
    got = oracle.prefill(q, wl.k_pool, wl.v_pool, wl.pre_bt, r)
    _, v = wl.logical_kv(wl.pre_bt, 40)
    v = W.bf16_bits_to_f32(v).astype(np.float64)
    for i in range(5):
        for h in range(4):
            want = v[: r + i + 1, h // 2, :].mean(axis=0)
            assert np.max(np.abs(got[i, h] - want)) <= 1e-13


def test_single_visible_key_returns_its_value_exactly():
    wl = _tiny_pool(8, 2, 128, 16, 20, seed=3)
    got = oracle.prefill(wl.q_pre[:1], wl.k_pool, wl.v_pool, wl.pre_bt, 0)
    _, v = wl.logical_kv(wl.pre_bt, 1)
    v = W.bf16_bits_to_f32(v).astype(np.float64)
    for h in range(8):
        assert np.array_equal(got[0, h], v[0, h // 4])


def test_constant_values_give_that_constant():
    wl = _tiny_pool(4, 1, 16, 4, 23, seed=5)
    vpool = np.full_like(wl.v_pool, W.f32_to_bf16_bits(np.float32(-1.375)))
    got = oracle.prefill(wl.q_pre[10:23], wl.k_pool, vpool, wl.pre_bt, 10)
    assert np.max(np.abs(got + 1.375)) <= 1e-14


def test_two_keys_give_logistic_weights():
    # q = a e_0 and k_j = b_j e_0, so s_j = scale * a * b_j; with two keys the
    # weight of key 1 is 1 / (1 + exp(s_0 - s_1)).
    d, page = 16, 4
    wl = _tiny_pool(1, 1, d, page, 2, seed=1)
    kp = np.zeros_like(wl.k_pool)
    vp = np.zeros_like(wl.v_pool)
    p0, p1 = wl.pre_bt[0], wl.pre_bt[0]
    kp[p0, 0, 0, 0] = W.f32_to_bf16_bits(np.float32(1.5))
    kp[p1, 0, 1, 0] = W.f32_to_bf16_bits(np.float32(-0.5))
    vp[p0, 0, 0, :] = W.f32_to_bf16_bits(np.float32(2.0))
    vp[p1, 0, 1, :] = W.f32_to_bf16_bits(np.float32(-4.0))
    q = np.zeros((1, 1, d), dtype=np.uint16)
    q[0, 0, 0] = W.f32_to_bf16_bits(np.float32(3.0))
    scale = 0.25
    got = oracle.prefill(q, kp, vp, wl.pre_bt, 1, scale=scale)  # row sees keys 0, 1
    s0, s1 = scale * 3.0 * 1.5, scale * 3.0 * -0.5
    w1 = 1.0 / (1.0 + math.exp(s0 - s1))
    want = (1 - w1) * 2.0 + w1 * -4.0
    assert np.max(np.abs(got[0, 0] - want)) <= 1e-14


def test_worked_example_fixture():
    with open(os.path.join(GOLDEN, "worked_example.json")) as f:
        ex = json.load(f)
    to16 = lambda a: W.f32_to_bf16_bits(np.asarray(a, dtype=np.float32))
    kp = to16(ex["k_pool"])
    vp = to16(ex["v_pool"])
    q = to16(ex["q"])
    assert np.array_equal(W.bf16_bits_to_f32(kp), np.asarray(ex["k_pool"], np.float32))
    bt = np.asarray(ex["block_table"], dtype=np.int32)
    got = oracle.paged_attention(q, kp, vp, bt, [0] * len(ex["nvis"]), ex["nvis"],
                                 scale=ex["scale"])
    e = math.e
    # closed forms derived in the fixture's "derivation" field
    want = np.array([[[(1 + e * e) / (1 + e + e * e), (e + e * e) / (1 + e + e * e)]],
                     [[1.0 / (1 + e), e / (1 + e)]]])
    assert np.max(np.abs(got - want)) <= 1e-15


def _permute_pages(wl: W.Workload, seed: int):
    """Relabel physical pages: the same logical content under another layout."""
    rng = np.random.default_rng(seed)
    P = wl.num_pages
    new_of_old = rng.permutation(P).astype(np.int32)
    kp = np.empty_like(wl.k_pool)
    vp = np.empty_like(wl.v_pool)
    kp[new_of_old] = wl.k_pool
    vp[new_of_old] = wl.v_pool
    return kp, vp, new_of_old[wl.pre_bt], new_of_old[wl.dec_bt]


def test_page_permutation_invariance_bit_exact():
    cfg = W.custom_config(hq=4, hkv=2, pre_chunks=((13, 30),), dec_batch=4,
                          dec_len_lo=1, dec_len_hi=90, seed=11)
    wl = W.make_workload(cfg)
    a = oracle.prefill(wl.q_pre[13:43], wl.k_pool, wl.v_pool, wl.pre_bt, 13)
    da = oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens)
    kp, vp, pbt, dbt = _permute_pages(wl, 99)
    b = oracle.prefill(wl.q_pre[13:43], kp, vp, pbt, 13)
    db = oracle.decode(wl.q_dec, kp, vp, dbt, wl.dec_lens)
    assert np.array_equal(a, b) and np.array_equal(da, db)


def test_chunked_prefill_equals_unchunked_bit_exact():
    wl = _tiny_pool(4, 2, 128, 16, 70, seed=2)
    full = oracle.prefill(wl.q_pre[:70], wl.k_pool, wl.v_pool, wl.pre_bt, 0)
    for r, n in ((0, 20), (20, 33), (53, 17)):
        part = oracle.prefill(wl.q_pre[r:r + n], wl.k_pool, wl.v_pool, wl.pre_bt, r)
        assert np.array_equal(part, full[r:r + n])


def test_future_keys_do_not_change_earlier_rows():
    wl = _tiny_pool(4, 2, 128, 16, 50, seed=4)
    a = oracle.prefill(wl.q_pre[:50], wl.k_pool, wl.v_pool, wl.pre_bt, 0)
    kp, vp = wl.k_pool.copy(), wl.v_pool.copy()
    cut = 31                                    # perturb keys at positions > 30
    for t in range(cut, 50):
        page, slot = wl.pre_bt[t // 16], t % 16
        kp[page, :, slot, :] ^= 0x1234
        vp[page, :, slot, :] ^= 0x0101
    b = oracle.prefill(wl.q_pre[:50], kp, vp, wl.pre_bt, 0)
    assert np.array_equal(a[:cut], b[:cut])
    assert not np.array_equal(a[cut:], b[cut:])


def test_decode_equals_last_prefill_row_bit_exact():
    wl = _tiny_pool(8, 2, 128, 16, 45, seed=6)
    for L in (1, 16, 17, 45):
        pre = oracle.prefill(wl.q_pre[L - 1:L], wl.k_pool, wl.v_pool, wl.pre_bt, L - 1)
        dec = oracle.decode(wl.q_pre[L - 1:L], wl.k_pool, wl.v_pool, wl.pre_bt[None, :], [L])
        assert np.array_equal(pre, dec)


def test_gqa_equals_mha_with_repeated_kv_bit_exact():
    wl = _tiny_pool(8, 2, 128, 16, 37, seed=8)
    g = 4
    kp = np.repeat(wl.k_pool, g, axis=1)        # kv head h // g becomes head h
    vp = np.repeat(wl.v_pool, g, axis=1)
    a = oracle.prefill(wl.q_pre[5:37], wl.k_pool, wl.v_pool, wl.pre_bt, 5)
    b = oracle.prefill(wl.q_pre[5:37], kp, vp, wl.pre_bt, 5)
    assert np.array_equal(a, b)


def test_thread_count_does_not_change_result():
    cfg = W.custom_config(hq=8, hkv=2, pre_chunks=((0, 9),), dec_batch=6,
                          dec_len_lo=1, dec_len_hi=120, seed=12)
    wl = W.make_workload(cfg)
    a = oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens, n_threads=1)
    b = oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens, n_threads=7)
    assert np.array_equal(a, b)


def test_softmax_weights_sum_to_one_and_respect_the_mask():
    wl = _tiny_pool(4, 2, 128, 16, 40, seed=9)
    _, p = oracle.prefill(wl.q_pre[10:40], wl.k_pool, wl.v_pool, wl.pre_bt, 10, want_probs=True)
    for i in range(30):
        nv = 10 + i + 1
        assert np.all(np.abs(p[i].sum(axis=-1) - 1.0) <= 1e-12)
        assert np.all(p[i][:, :nv] > 0) and np.all(p[i][:, nv:] == 0)


def test_doubling_values_doubles_output_exactly():
    wl = _tiny_pool(4, 2, 128, 16, 33, seed=10)
    a = oracle.prefill(wl.q_pre[:33], wl.k_pool, wl.v_pool, wl.pre_bt, 0)
    v2 = W.f32_to_bf16_bits(2 * W.bf16_bits_to_f32(wl.v_pool))
    b = oracle.prefill(wl.q_pre[:33], wl.k_pool, v2, wl.pre_bt, 0)
    assert np.array_equal(2 * a, b)


@pytest.mark.parametrize("cut", [0, 1, 16, 29, 57, 58])
def test_merge_of_parts_equals_whole(cut):
    wl = _tiny_pool(4, 2, 128, 16, 58, seed=13)
    q = wl.q_pre[57]
    whole = oracle.prefill(wl.q_pre[57:58], wl.k_pool, wl.v_pool, wl.pre_bt, 57)[0]
    for h in range(4):
        m0, l0, o0 = oracle.partial(q, wl.k_pool, wl.v_pool, wl.pre_bt, h, 0, cut)
        m1, l1, o1 = oracle.partial(q, wl.k_pool, wl.v_pool, wl.pre_bt, h, cut, 58)
        merged = oracle.merge_parts([m0, m1], [l0, l1], np.stack([o0, o1]))
        assert np.max(np.abs(merged - whole[h])) <= 1e-13


def test_oracle_rejects_pages_outside_the_pool():
    wl = _tiny_pool(4, 2, 128, 16, 20)
    bt = wl.pre_bt.copy()
    bt[1] = wl.num_pages                      # one past the end
    with pytest.raises(ValueError):
        oracle.prefill(wl.q_pre[:20], wl.k_pool, wl.v_pool, bt, 0)
    with pytest.raises(ValueError):            # more keys than the table maps
        oracle.decode(wl.q_pre[:1], wl.k_pool, wl.v_pool, wl.pre_bt[None, :2], [33])
