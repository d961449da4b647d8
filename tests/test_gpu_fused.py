"""The fused prefill + decode launch: every output bit-identical to the two
separate calls (same work-group bodies, same splits), and the small cases
against the oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2504_14489_amd import mw, workloads as W
from paper_2504_14489_amd.device import DeviceWorkload, Timing, to_bits
from tests.helpers import assert_close, say

pytestmark = pytest.mark.gpu

CASES = {
    # two contiguous chunks (a chunk over a cached prefix), ragged decode lengths
    "chunks": dict(hq=8, hkv=2, pre_chunks=((0, 200), (200, 180)), dec_batch=6, dec_len_lo=100, dec_len_hi=900),
    # an odd number of decode units (one work-group half idle), group of 1
    "odd_units": dict(hq=3, hkv=3, pre_chunks=((0, 70),), dec_batch=1, dec_len_lo=17, dec_len_hi=17),
    # many short decodes next to a one-token prefill
    "tiny_prefill": dict(hq=8, hkv=1, pre_chunks=((0, 1),), dec_batch=33, dec_len_lo=1, dec_len_hi=300),
    # GQA group 16 (the decode kernel's maximum), long prefill
    "group16": dict(hq=16, hkv=1, pre_chunks=((0, 700),), dec_batch=3, dec_len_lo=1000, dec_len_hi=2500),
}


def separate(dw, dec, pre, stream):
    # the fused call takes chunk_pages 0 as automatic fixed chunks (-1)
    ch = dec.get("chunk_pages", 0) or -1
    mw.mw_prefill_attn(pre["pool"], dw.hq, dw.hkv, dw.d, dw.scale, pre["new_lens"], pre["prefix_lens"],
                       pre["d_qo_indptr"], pre["d_prefix_lens"], pre["d_block_table"], pre["bt_stride"],
                       pre["d_q"], pre["d_out"], stream, None)
    mw.mw_decode_attn(dec["pool"], dw.hq, dw.hkv, dw.d, dw.scale, dw.dec_lens, dec["d_seq_lens"],
                      dec["d_block_table"], dec["bt_stride"], dec["d_q"], dec["d_out"], dec["d_workspace"],
                      dec["workspace_bytes"], ch, stream, None)
    mw.mw_sync(stream)
    return dw.o_pre.clone(), dw.o_dec.clone()


def fused(dw, dec, pre, stream):
    dw.o_pre.zero_()
    dw.o_dec.zero_()
    torch.cuda.synchronize()
    mw.mw_fused_attn(pre, dec, stream)
    mw.mw_sync(stream)
    return dw.o_pre.clone(), dw.o_dec.clone()


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("chunk_pages", [0, 8])
def test_fused_matches_separate_calls_and_oracle(name, chunk_pages):
    cfg = W.custom_config(name, **CASES[name])
    wl = W.make_workload(cfg, seed=5)
    say(f"fused {name} chunk_pages {chunk_pages}")
    dw = DeviceWorkload(wl)
    try:
        dec, pre = dw.engine_args(chunk_pages)
        s = torch.cuda.current_stream().cuda_stream
        ref_pre, ref_dec = separate(dw, dec, pre, s)
        got_pre, got_dec = fused(dw, dec, pre, s)
        n = cfg.pre_total
        assert torch.equal(got_pre[:n], ref_pre[:n]), "prefill differs from the separate call"
        assert torch.equal(got_dec, ref_dec), "decode differs from the separate call"
        assert_close(to_bits(got_pre[:n]), oracle.prefill(wl.q_pre[:n], wl.k_pool, wl.v_pool, wl.pre_bt, 0),
                     f"fused prefill {name}")
        assert_close(to_bits(got_dec), oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens),
                     f"fused decode {name}")
    finally:
        dw.close()


@pytest.mark.parametrize("config", ["llama8b", "llama70b"])
def test_fused_full_size_matches_separate_calls(config):
    """At full size the separate calls are the ones the oracle checks on
    sampled rows; the fused launch must reproduce them bit for bit, also on a
    CU-masked stream (block pairing depends on the stream's CUs)."""
    from paper_2504_14489_amd.device import Partition
    wl = W.make_workload(W.CONFIGS[config], seed=0)
    say(f"fused full size {config}")
    dw = DeviceWorkload(wl)
    part = Partition(128, 128)
    try:
        dec, pre = dw.engine_args()
        for s in (torch.cuda.current_stream().cuda_stream, part.prefill_stream):
            ref_pre, ref_dec = separate(dw, dec, pre, s)
            got_pre, got_dec = fused(dw, dec, pre, s)
            assert torch.equal(got_pre, ref_pre) and torch.equal(got_dec, ref_dec)
        t = Timing()
        mw.mw_fused_attn(pre, dec, part.prefill_stream, t.h)
        mw.mw_sync(part.prefill_stream)
        assert mw.mw_timing_kernels(t.h) == 2 and t.kernel_ms(0) > 0.0
        t.close()
    finally:
        part.close()
        dw.close()


def test_fused_rejects_mismatched_pools():
    cfg = W.custom_config("pools", **CASES["chunks"])
    wl = W.make_workload(cfg, seed=1)
    dw, dw2 = DeviceWorkload(wl), DeviceWorkload(wl)
    try:
        dec, _ = dw.engine_args()
        _, pre = dw2.engine_args()
        with pytest.raises(mw.MWError) as e:
            mw.mw_fused_attn(pre, dec, 0)
        assert e.value.status == mw.MW_ERR_INVALID_ARG
    finally:
        dw.close()
        dw2.close()
