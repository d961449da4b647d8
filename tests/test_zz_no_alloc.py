"""The decode entry point that allocates nothing (its workspace is the
library's static device array) against mw_decode_attn and the oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2504_14489_amd import mw
from paper_2504_14489_amd import workloads as W
from paper_2504_14489_amd.device import DeviceWorkload, Partition, to_bits
from tests.helpers import assert_close, say

pytestmark = pytest.mark.gpu


def noalloc_decode(dw, stream=0, chunk_pages=0):
    out = torch.zeros_like(dw.q_dec)
    torch.cuda.synchronize()
    mw.mw_decode_attn_noalloc(dw.pool, dw.hq, dw.hkv, dw.d, dw.scale, dw.dec_lens, dw.d_dec_lens.data_ptr(),
                              dw.dec_bt.data_ptr(), dw.dec_bt.shape[1], dw.q_dec.data_ptr(), out.data_ptr(),
                              chunk_pages, stream)
    return out


@pytest.mark.parametrize("chunk_pages", [0, -1])
def test_noalloc_decode_equals_the_workspace_call_twice_in_a_row(chunk_pages):
    """Two calls in a row, the second on a smaller batch (the array keeps the
    first call's partials), then two long sequences (whose segments the
    balanced split pads to whole ranges), each bit-equal to mw_decode_attn
    with a caller workspace on the same stream, and within tolerance of the
    oracle."""
    part = Partition(64, 192)
    try:
        for name, cfg, lens in (("llama8b", W.CONFIGS["llama8b"], None),
                                ("small", W.custom_config(hq=32, hkv=8, pre_chunks=((0, 1),), dec_batch=9,
                                                          dec_len_lo=1, dec_len_hi=700, seed=12), None),
                                ("two_long", W.custom_config(hq=32, hkv=8, pre_chunks=((0, 1),), dec_batch=2,
                                                             seed=13), [20000, 15000])):
            say(f"noalloc decode {name} chunk_pages={chunk_pages}")
            wl = W.make_workload(cfg, dec_lens=lens) if lens else W.make_workload(cfg)
            dw = DeviceWorkload(wl)
            try:
                got = to_bits(noalloc_decode(dw, part.decode_stream, chunk_pages))
                want = to_bits(dw.decode(part.decode_stream, chunk_pages=chunk_pages))
                torch.cuda.synchronize()
            finally:
                dw.close()
            assert np.array_equal(got, want), f"{name}: differs from mw_decode_attn"
            ref = oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens)
            assert_close(got, ref, f"noalloc decode {name}")
    finally:
        part.close()


def test_noalloc_decode_rejects_calls_beyond_the_scratch_size():
    """4096 one-token sequences over 8 kv heads with 16 query heads each need
    far more than 16 MiB of partials: refused before anything is launched."""
    say("noalloc decode oversized call")
    dev = torch.device("cuda:0")
    B, hkv, hq = 4096, 8, 128
    kp = torch.zeros(2 * hkv * 16 * 128, dtype=torch.int16, device=dev)
    vp = torch.zeros_like(kp)
    q = torch.zeros(B * hq * 128, dtype=torch.int16, device=dev)
    out = torch.zeros_like(q)
    lens = np.ones(B, np.int32)
    d_lens = torch.ones(B, dtype=torch.int32, device=dev)
    bt = torch.zeros(B, dtype=torch.int32, device=dev)
    pool = mw.mw_kv_pool_create(2, 16, hkv, 128, kp.data_ptr(), vp.data_ptr())
    try:
        need = mw.mw_decode_workspace_size(hq, hkv, 128, lens, 0)
        assert need > 16 << 20
        with pytest.raises(mw.MWError) as e:
            mw.mw_decode_attn_noalloc(pool, hq, hkv, 128, 128 ** -0.5, lens, d_lens.data_ptr(), bt.data_ptr(), 1,
                                      q.data_ptr(), out.data_ptr())
        assert e.value.status == mw.MW_ERR_UNSUPPORTED and "static scratch" in e.value.message
        torch.cuda.synchronize()
        assert not out.any(), "a refused call wrote output"
    finally:
        mw.mw_kv_pool_destroy(pool)
