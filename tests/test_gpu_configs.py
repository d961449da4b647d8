"""Every workload at its full size on the GPU, against the oracle on sampled
rows (the oracle computes those rows one by one) plus properties that hold at
any size (every output finite; multiplexed equals isolated bit for bit)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2504_14489_amd import workloads as W
from paper_2504_14489_amd.device import DeviceWorkload, Partition, to_bits
from tests.helpers import assert_close, say

pytestmark = pytest.mark.gpu


def sample_rows(n, k=12):
    """First, last, tile and page boundaries, and evenly spread rows."""
    idx = {0, 1, 15, 16, 63, 64, 65, n // 2, n - 2, n - 1}
    idx |= set(np.linspace(0, n - 1, k).astype(int).tolist())
    return sorted(i for i in idx if 0 <= i < n)


def sample_seqs(lens, k=6):
    order = np.argsort(lens, kind="stable")
    idx = {int(order[0]), int(order[-1]), int(order[len(order) // 2])}
    idx |= set(np.linspace(0, len(lens) - 1, k).astype(int).tolist())
    return sorted(idx)


@pytest.mark.parametrize("name", ["llama8b", "llama70b", "llama70b_tp8", "longctx8b", "sweep8b"])
def test_full_size_config(name):
    cfg = W.CONFIGS[name]
    say(f"full-size {name}: generating")
    wl = W.make_workload(cfg)
    dw = DeviceWorkload(wl)
    part = Partition(cfg.prefill_cus[0], cfg.decode_cus[0])
    try:
        say(f"full-size {name}: isolated then multiplexed runs")
        for r, n in cfg.pre_chunks:
            dw.prefill(r, n, part.prefill_stream)
        dw.decode(part.decode_stream)
        torch.cuda.synchronize()
        iso_pre, iso_dec = to_bits(dw.o_pre), to_bits(dw.o_dec)
        dw.o_pre.zero_(); dw.o_dec.zero_()
        torch.cuda.synchronize()
        dw.decode(part.decode_stream)              # decode first, then prefill
        for r, n in cfg.pre_chunks:
            dw.prefill(r, n, part.prefill_stream)
        torch.cuda.synchronize()
        got_pre, got_dec = to_bits(dw.o_pre), to_bits(dw.o_dec)
    finally:
        part.close()
        dw.close()
    assert np.array_equal(iso_pre, got_pre) and np.array_equal(iso_dec, got_dec), \
        "multiplexed outputs differ from isolated ones"
    assert np.all(np.isfinite(W.bf16_bits_to_f32(got_pre[:wl.pre_len])))
    assert np.all(np.isfinite(W.bf16_bits_to_f32(got_dec)))
    for r, n in cfg.pre_chunks:
        rows = sample_rows(n)
        say(f"full-size {name}: oracle on {len(rows)} rows of chunk r={r} n={n}")
        ref = np.concatenate([oracle.prefill(wl.q_pre[r + i:r + i + 1], wl.k_pool, wl.v_pool,
                                             wl.pre_bt, r + i) for i in rows])
        assert_close(got_pre[[r + i for i in rows]], ref, f"{name} prefill r={r}")
    seqs = sample_seqs(wl.dec_lens)
    say(f"full-size {name}: oracle on decode sequences {seqs}")
    ref = oracle.decode(wl.q_dec[seqs], wl.k_pool, wl.v_pool, wl.dec_bt[seqs], wl.dec_lens[seqs])
    assert_close(got_dec[seqs], ref, f"{name} decode")


def test_tiny_config_multiplexed_full_parity():
    cfg = W.CONFIGS["tiny"]
    wl = W.make_workload(cfg)
    dw = DeviceWorkload(wl)
    part = Partition(128, 128)
    try:
        dw.decode(part.decode_stream)
        dw.prefill(0, 256, part.prefill_stream)
        torch.cuda.synchronize()
        got_pre, got_dec = to_bits(dw.o_pre), to_bits(dw.o_dec)
    finally:
        part.close()
        dw.close()
    assert_close(got_pre, oracle.prefill(wl.q_pre, wl.k_pool, wl.v_pool, wl.pre_bt, 0), "tiny prefill")
    assert_close(got_dec, oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens),
                 "tiny decode")
