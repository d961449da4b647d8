"""Causal prefill attention on the GPU against the CPU oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2504_14489_amd import workloads as W
from paper_2504_14489_amd import mw
from paper_2504_14489_amd.device import DeviceWorkload, Partition, Timing, to_bits
from tests.helpers import assert_close, say

pytestmark = pytest.mark.gpu

# (prefix r, new n): empty prefix, single token, tile and page boundaries, ragged tails
CHUNKS = [(0, 1), (0, 63), (0, 64), (0, 65), (5, 100), (33, 17), (100, 130), (0, 256),
          (64, 64), (1, 200)]


def run_prefill(wl, r, n):
    dw = DeviceWorkload(wl)
    try:
        o = dw.prefill(r, n)
        torch.cuda.synchronize()
        return to_bits(o)
    finally:
        dw.close()


@pytest.mark.parametrize("hq,hkv", [(8, 2), (64, 8), (4, 4), (2, 1), (12, 2)])
@pytest.mark.parametrize("q_scale", [1.0, 4.0])
def test_prefill_matches_oracle(hq, hkv, q_scale):
    for r, n in CHUNKS:
        say(f"prefill hq={hq} hkv={hkv} r={r} n={n} q_scale={q_scale}")
        cfg = W.custom_config(hq=hq, hkv=hkv, pre_chunks=((r, n),), dec_batch=1, dec_len_lo=1,
                              dec_len_hi=2, seed=r * 7 + n)
        wl = W.make_workload(cfg, q_scale=q_scale)
        got = run_prefill(wl, r, n)
        ref = oracle.prefill(wl.q_pre[r:r + n], wl.k_pool, wl.v_pool, wl.pre_bt, r)
        assert_close(got, ref, f"prefill hq={hq} hkv={hkv} r={r} n={n}")


def test_prefill_tiny_config_full_parity():
    say("prefill tiny config")
    wl = W.make_workload(W.CONFIGS["tiny"])
    got = run_prefill(wl, 0, 256)
    ref = oracle.prefill(wl.q_pre[:256], wl.k_pool, wl.v_pool, wl.pre_bt, 0)
    assert_close(got, ref, "prefill tiny")


def test_chunked_prefill_matches_unchunked():
    say("prefill chunked vs unchunked")
    cfg = W.custom_config(hq=8, hkv=2, pre_chunks=((0, 300),), dec_batch=1, dec_len_lo=1,
                          dec_len_hi=2, seed=3)
    wl = W.make_workload(cfg)
    dw = DeviceWorkload(wl)
    try:
        full = to_bits(dw.prefill(0, 300).clone())
        parts = [to_bits(dw.prefill(r, n).clone()) for r, n in ((0, 100), (100, 77), (177, 123))]
        torch.cuda.synchronize()
    finally:
        dw.close()
    chunked = np.concatenate(parts)
    ref = oracle.prefill(wl.q_pre[:300], wl.k_pool, wl.v_pool, wl.pre_bt, 0)
    assert_close(full, ref, "unchunked")
    assert_close(chunked, ref, "chunked")


def test_prefill_page_permutation_invariance_and_determinism():
    say("prefill permutation invariance")
    cfg = W.custom_config(hq=8, hkv=2, pre_chunks=((40, 150),), dec_batch=1, dec_len_lo=1,
                          dec_len_hi=2, seed=9)
    wl = W.make_workload(cfg)
    a = run_prefill(wl, 40, 150)
    assert np.array_equal(a, run_prefill(wl, 40, 150)), "run-to-run results differ"
    rng = np.random.default_rng(5)
    new_of_old = rng.permutation(wl.num_pages).astype(np.int32)
    k = np.empty_like(wl.k_pool); k[new_of_old] = wl.k_pool
    v = np.empty_like(wl.v_pool); v[new_of_old] = wl.v_pool
    wl2 = W.Workload(cfg=wl.cfg, k_pool=k, v_pool=v, nan_page=int(new_of_old[wl.nan_page]),
                     pre_len=wl.pre_len, pre_bt=new_of_old[wl.pre_bt], q_pre=wl.q_pre,
                     dec_lens=wl.dec_lens, dec_bt=new_of_old[wl.dec_bt], q_dec=wl.q_dec,
                     perm=wl.perm)
    assert np.array_equal(a, run_prefill(wl2, 40, 150)), "page renumbering changed the result"


def _varlen_setup(seqs, hq, hkv, seed0):
    """One pool holding every sequence's pages (the workloads' pools laid end
    to end, tables offset), their block-table rows, and the batch's Q rows."""
    cfgs = [W.custom_config(hq=hq, hkv=hkv, pre_chunks=((r, n),), dec_batch=1, dec_len_lo=1,
                            dec_len_hi=2, seed=seed0 + i) for i, (r, n) in enumerate(seqs)]
    wls = [W.make_workload(c) for c in cfgs]
    k = np.concatenate([w.k_pool for w in wls]); v = np.concatenate([w.v_pool for w in wls])
    offs = np.cumsum([0] + [w.num_pages for w in wls])
    stride = max(len(w.pre_bt) for w in wls)
    bt = np.full((len(seqs), stride), 0, np.int32)
    for i, w in enumerate(wls):
        bt[i, :len(w.pre_bt)] = w.pre_bt + offs[i]
    q = np.concatenate([w.q_pre[r:r + n] for w, (r, n) in zip(wls, seqs)])
    return wls, k, v, bt, stride, q


def test_prefill_varlen_batch():
    """Three sequences in one call (block-table rows, varlen Q/O offsets)."""
    say("prefill varlen batch")
    from paper_2504_14489_amd import mw
    seqs = [(0, 70), (20, 5), (130, 64)]
    wls, k, v, bt, stride, q = _varlen_setup(seqs, 8, 2, 40)
    dev = torch.device("cuda:0")
    t16 = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev)
    t32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)
    dk, dv, dq, dbt = t16(k), t16(v), t16(q), t32(bt)
    do = torch.zeros_like(dq)
    indptr = t32(np.cumsum([0] + [n for _, n in seqs]))
    pref = t32([r for r, _ in seqs])
    pool = mw.mw_kv_pool_create(k.shape[0], 16, 2, 128, dk.data_ptr(), dv.data_ptr())
    try:
        mw.mw_prefill_attn(pool, 8, 2, 128, 1 / np.sqrt(128), [n for _, n in seqs],
                           [r for r, _ in seqs], indptr.data_ptr(), pref.data_ptr(),
                           dbt.data_ptr(), stride, dq.data_ptr(), do.data_ptr())
        torch.cuda.synchronize()
    finally:
        mw.mw_kv_pool_destroy(pool)
    got = to_bits(do)
    row = 0
    for w, (r, n) in zip(wls, seqs):
        ref = oracle.prefill(w.q_pre[r:r + n], w.k_pool, w.v_pool, w.pre_bt, r)
        assert_close(got[row:row + n], ref, f"varlen seq r={r} n={n}")
        row += n


def test_prefill_varlen_batch_with_the_split_on_partitions():
    """Four sequences of different prefixes and lengths in one call, through
    the split-enabled entry point on 8 and 96 CUs and the whole GPU (the plan
    cuts the long-prefix sequence's blocks into key ranges), and through the
    plain one: every row against the oracle, and the plain and split calls
    within the tolerance of each other."""
    from paper_2504_14489_amd import mw
    from paper_2504_14489_amd.device import Partition
    hq, hkv = 8, 2
    seqs = [(0, 700), (5000, 90), (300, 1500), (12000, 33)]
    say(f"prefill varlen batch with the split: {seqs}")
    wls, k, v, bt, stride, q = _varlen_setup(seqs, hq, hkv, 60)
    dev = torch.device("cuda:0")
    t16 = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev)
    t32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)
    dk, dv, dq, dbt = t16(k), t16(v), t16(q), t32(bt)
    ns, rs = [n for _, n in seqs], [r for r, _ in seqs]
    indptr, pref = t32(np.cumsum([0] + ns)), t32(rs)
    pool = mw.mw_kv_pool_create(k.shape[0], 16, hkv, 128, dk.data_ptr(), dv.data_ptr())
    results, cut = {}, {}
    try:
        for cus in (8, 96, 0):
            part = Partition(cus, 256 - cus) if cus else None
            stream = part.prefill_stream if part else 0
            try:
                nbytes = mw.mw_prefill_workspace_size(hq, hkv, 128, ns, rs, cus or 256)
                ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=dev)
                for split in (True, False):
                    do = torch.zeros_like(dq)
                    t = Timing()
                    if split:
                        mw.mw_prefill_attn_ws(pool, hq, hkv, 128, 1 / np.sqrt(128), ns, rs, indptr.data_ptr(),
                                              pref.data_ptr(), dbt.data_ptr(), stride, dq.data_ptr(), do.data_ptr(),
                                              ws.data_ptr(), ws.numel(), stream, t.h)
                    else:
                        mw.mw_prefill_attn(pool, hq, hkv, 128, 1 / np.sqrt(128), ns, rs, indptr.data_ptr(),
                                           pref.data_ptr(), dbt.data_ptr(), stride, dq.data_ptr(), do.data_ptr(),
                                           stream, t.h)
                    torch.cuda.synchronize()
                    results[(cus, split)] = to_bits(do).copy()
                    if split:
                        cut[cus] = (mw.mw_timing_kernels(t.h) == 2, nbytes > 0)
                    t.close()
            finally:
                if part:
                    part.close()
    finally:
        mw.mw_kv_pool_destroy(pool)
    for cus, (two_kernels, planned) in cut.items():
        assert two_kernels == planned, f"{cus} CUs: the call and the workspace size disagree on the cut"
    assert any(planned for _, planned in cut.values()), "no partition cut the batch"
    refs = [oracle.prefill(w.q_pre[r:r + n], w.k_pool, w.v_pool, w.pre_bt, r) for w, (r, n) in zip(wls, seqs)]
    for (cus, split), got in results.items():
        row = 0
        for ref, (r, n) in zip(refs, seqs):
            assert_close(got[row:row + n], ref, f"varlen r={r} n={n} on {cus or 'all'} CUs, split={split}")
            row += n


def test_prefill_same_result_on_any_cu_count():
    """The launch pairs heavy and light query blocks only when the pairs fill
    whole rounds of the stream's CUs, and uses 4-wave work-groups on 32-position
    blocks when the 8-wave pairs would not give every CU one (here: paired
    8-wave blocks on 32 CUs, single 4-wave blocks on 64 and on all CUs); every
    such choice must give the same bits (the plain call: the key-range split,
    which changes rounding, is tested on its own)."""
    say("prefill split independence (32 / 64 / all CUs)")
    from paper_2504_14489_amd.device import Partition
    cfg = W.custom_config(hq=32, hkv=8, pre_chunks=((0, 512),), dec_batch=1, dec_len_lo=1,
                          dec_len_hi=2, seed=21)
    wl = W.make_workload(cfg)
    dw = DeviceWorkload(wl)
    outs = []
    try:
        for p_cus in (32, 64, 0):  # 32 pairs: paired on 32 CUs, single blocks otherwise
            part = Partition(p_cus, 256 - p_cus) if p_cus else None
            try:
                o = dw.prefill(0, 512, part.prefill_stream if part else 0, split=False)
                torch.cuda.synchronize()
                outs.append(to_bits(o))
            finally:
                if part:
                    part.close()
    finally:
        dw.close()
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2]), "split changed the result"
    rows = [0, 63, 64, 255, 511]
    ref = oracle.prefill(wl.q_pre[:512], wl.k_pool, wl.v_pool, wl.pre_bt, 0)
    assert_close(outs[0][rows], ref[rows], "split independence rows")


def _scale_keys(wl, bt, positions, factor):
    """Multiplies the K rows of the given logical positions (all kv heads) by a
    power of two, exactly in bf16."""
    from paper_2504_14489_amd.device import bits_to_f32
    k = wl.k_pool.copy()
    for t in positions:
        page, slot = bt[t // 16], t % 16
        row = bits_to_f32(k[page, :, slot, :]) * factor
        k[page, :, slot, :] = (row.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    return W.Workload(cfg=wl.cfg, k_pool=k, v_pool=wl.v_pool, nan_page=wl.nan_page, pre_len=wl.pre_len,
                      pre_bt=wl.pre_bt, q_pre=wl.q_pre, dec_lens=wl.dec_lens, dec_bt=wl.dec_bt,
                      q_dec=wl.q_dec, perm=wl.perm)


def test_prefill_wide_score_range():
    """A few keys scaled by 32 against Q scaled by 8 spread the scaled scores
    over hundreds of log2 units, with the largest in either half of a
    score accumulator's lanes: the running maximum must cover both halves (a
    reference taken from half the keys overflows 2^(s - m)), and the late large
    keys force the lazy rescale."""
    say("prefill wide score range")
    cfg = W.custom_config(hq=8, hkv=2, pre_chunks=((0, 200),), dec_batch=1, dec_len_lo=1,
                          dec_len_hi=2, seed=77)
    wl = _scale_keys(W.make_workload(cfg, q_scale=8.0), W.make_workload(cfg).pre_bt,
                     [4, 5, 70, 131, 150, 199], 32.0)
    got = run_prefill(wl, 0, 200)
    ref = oracle.prefill(wl.q_pre[:200], wl.k_pool, wl.v_pool, wl.pre_bt, 0)
    assert_close(got, ref, "prefill wide score range")


def test_empty_batches_and_zero_length_sequences():
    """Degenerate inputs: no sequences at all, and a zero-length sequence next
    to a real one in one varlen call (its rows are absent, the other's are
    exact); nothing is launched for an empty call."""
    say("prefill/decode empty and zero-length inputs")
    from paper_2504_14489_amd import mw
    cfg = W.custom_config(hq=8, hkv=2, pre_chunks=((0, 40),), dec_batch=1, dec_len_lo=1, dec_len_hi=2, seed=77)
    wl = W.make_workload(cfg)
    dw = DeviceWorkload(wl)
    try:
        dev = dw.device
        t32 = lambda a: torch.from_numpy(np.asarray(a, dtype=np.int32)).to(dev)
        # batch 0: both phases return without launching
        mw.mw_prefill_attn(dw.pool, 8, 2, 128, dw.scale, [], [], 0, 0, 0, 1, 0, 0)
        nbytes = mw.mw_decode_workspace_size(8, 2, 128, [], 0)
        ws = torch.zeros(max(nbytes, 16), dtype=torch.uint8, device=dev)
        mw.mw_decode_attn(dw.pool, 8, 2, 128, dw.scale, [], 0, 0, 1, 0, 0, ws.data_ptr(), ws.numel())
        # a zero-length sequence before a 40-token one, sharing the block table
        bt = t32(np.stack([wl.pre_bt, wl.pre_bt]))
        indptr, pref = t32([0, 0, 40]), t32([0, 0])
        out = torch.zeros_like(dw.q_pre)
        mw.mw_prefill_attn(dw.pool, 8, 2, 128, dw.scale, [0, 40], [0, 0], indptr.data_ptr(), pref.data_ptr(),
                           bt.data_ptr(), bt.shape[1], dw.q_pre.data_ptr(), out.data_ptr())
        torch.cuda.synchronize()
        ref = oracle.prefill(wl.q_pre[:40], wl.k_pool, wl.v_pool, wl.pre_bt, 0)
        assert_close(to_bits(out[:40]), ref, "zero-length neighbour")
    finally:
        dw.close()


SLACKS = [(W.BF16_NAN, W.BF16_NAN), (W.BF16_POS_INF, W.BF16_NEG_INF), (W.BF16_NAN, W.BF16_POS_INF)]


@pytest.mark.parametrize("slack", SLACKS, ids=["nan-nan", "inf-neginf", "nan-inf"])
def test_prefill_ignores_nan_and_inf_in_slack_slots(slack):
    """Slots past a sequence's end in its last page may hold any bits: a key
    there is masked (p = 0), and its value must never be read, since 0 * NaN
    and 0 * Inf are NaN.  Ragged lengths on the whole GPU (4-wave blocks) and
    on 8 CUs (8-wave paired blocks for the largest case)."""
    from paper_2504_14489_amd.device import Partition
    cases = [((0, 1), 8, 2), ((5, 100), 8, 2), ((33, 17), 32, 8), ((100, 130), 16, 1), ((0, 509), 32, 8)]
    part = Partition(8, 8)
    try:
        for (r, n), hq, hkv in cases:
            say(f"prefill slack {slack} hq={hq} hkv={hkv} r={r} n={n}")
            cfg = W.custom_config(hq=hq, hkv=hkv, pre_chunks=((r, n),), dec_batch=1, dec_len_lo=1,
                                  dec_len_hi=2, seed=r + 3 * n)
            wl = W.make_workload(cfg, slack_bits=slack)
            assert (r + n) % 16, "the case must leave slack in its last page"
            ref = oracle.prefill(wl.q_pre[r:r + n], wl.k_pool, wl.v_pool, wl.pre_bt, r)
            dw = DeviceWorkload(wl)
            try:
                for stream in (0, part.prefill_stream):
                    o = dw.prefill(r, n, stream)
                    torch.cuda.synchronize()
                    assert_close(to_bits(o), ref, f"prefill slack r={r} n={n} stream={'all' if stream == 0 else 8}")
            finally:
                dw.close()
    finally:
        part.close()


def test_prefill_block_table_longer_than_the_lds_copy():
    """A sequence of more than 4096 pages (65,536 tokens): the work-group's
    copy of its block table in LDS holds the first 4096 entries and the rest
    are read from global memory.  130 new tokens over a 70,001-token prefix
    with one kv head: 4-wave blocks on the whole GPU (plain, and cut into key
    ranges by the split, each piece's table copy starting at its first page),
    8-wave paired blocks on 8 CUs; every row against the oracle."""
    from paper_2504_14489_amd.device import Partition
    r, n = 70001, 130
    say(f"prefill long block table r={r} n={n}")
    cfg = W.custom_config(hq=16, hkv=1, pre_chunks=((r, n),), dec_batch=1, dec_len_lo=1, dec_len_hi=2,
                          seed=70)
    wl = W.make_workload(cfg)
    assert len(wl.pre_bt) > 4096
    dw = DeviceWorkload(wl)
    part = Partition(8, 8)
    outs = []
    try:
        for stream, split in ((0, False), (part.prefill_stream, False), (0, True)):
            t = Timing()
            o = dw.prefill(r, n, stream, t.h, split=split)
            torch.cuda.synchronize()
            outs.append(to_bits(o).copy())
            kernels = mw.mw_timing_kernels(t.h)
            t.close()
    finally:
        part.close()
        dw.close()
    assert kernels == 2, "the whole-GPU call with a workspace did not split"
    ref = oracle.prefill(wl.q_pre[r:r + n], wl.k_pool, wl.v_pool, wl.pre_bt, r)
    for o, where in zip(outs, ("whole GPU", "8 CUs", "whole GPU, key-range split")):
        mx, mean = assert_close(o, ref, f"long table on {where}")
        say(f"  {where}: max-abs {mx:.3g} mean-abs {mean:.3g}")
    assert np.array_equal(outs[0], outs[1]), "4-wave and 8-wave launches differ"


# (prefix r, new n, q heads, kv heads, CUs of the stream (0: all), the plan
# must cut): causal blocks long enough to be cut into key ranges, ragged
# tails, a GQA group of 6 (idle waves in the second head group), a
# one-kv-head shard of a 70B-shaped layer (2048-token chunks: the first on the
# whole GPU, the last on 96 CUs), and calls the plan may keep whole (short
# blocks on 96 CUs, a grid of two blocks per CU, one 5-tile block)
SPLIT_CASES = [(1000, 130, 8, 2, 0, True), (333, 257, 12, 2, 0, True), (0, 2048, 8, 1, 0, True),
               (6144, 2048, 8, 1, 96, True), (4100, 33, 4, 1, 0, True), (0, 1000, 8, 2, 0, True),
               (0, 2048, 8, 1, 96, False), (0, 1000, 32, 8, 0, False), (257, 1, 8, 1, 0, False)]


@pytest.mark.parametrize("r,n,hq,hkv,cus,must_cut", SPLIT_CASES)
def test_prefill_key_range_split(r, n, hq, hkv, cus, must_cut):
    """Prefill with the key-range split (pieces of each causal block's keys,
    merged by log-sum-exp) against the oracle on every row.  The call splits
    exactly when the workspace size for the stream's CU count says the plan
    cuts, and the result is the same from run to run."""
    say(f"prefill key-range split r={r} n={n} hq={hq} hkv={hkv} cus={cus or 'all'}")
    cfg = W.custom_config(hq=hq, hkv=hkv, pre_chunks=((r, n),), dec_batch=1, dec_len_lo=1, dec_len_hi=2,
                          seed=r + 3 * n)
    wl = W.make_workload(cfg)
    dw = DeviceWorkload(wl)
    part = Partition(cus, 256 - cus) if cus else None
    stream = part.prefill_stream if part else 0
    outs, kernels = [], []
    try:
        for _ in range(2):
            t = Timing()
            o = dw.prefill(r, n, stream, t.h)
            torch.cuda.synchronize()
            outs.append(to_bits(o).copy())
            kernels.append(mw.mw_timing_kernels(t.h))
            t.close()
    finally:
        if part:
            part.close()
        dw.close()
    assert np.array_equal(outs[0], outs[1]), "run-to-run results differ"
    planned = mw.mw_prefill_workspace_size(hq, hkv, 128, [n], [r], cus or 256) > 0
    assert planned or not must_cut, "the plan does not cut"
    assert (kernels[0] == 2) == planned, f"{kernels[0]} kernel(s), plan cuts: {planned}"
    ref = oracle.prefill(wl.q_pre[r:r + n], wl.k_pool, wl.v_pool, wl.pre_bt, r)
    mx, mean = assert_close(outs[0], ref, f"split r={r} n={n}")
    say(f"  {kernels[0]} kernel(s): max-abs {mx:.3g} mean-abs {mean:.3g}")
