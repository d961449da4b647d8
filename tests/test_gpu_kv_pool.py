"""KV append and gather on the GPU are bit copies through the block table."""
import numpy as np
import pytest
import torch

from paper_2504_14489_amd import workloads as W
from paper_2504_14489_amd.device import DeviceWorkload, to_bits, _dev16
from paper_2504_14489_amd import mw
from tests.helpers import say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("r,n", [(0, 1), (0, 16), (5, 30), (31, 97), (100, 1)])
def test_prefill_append_is_bit_exact(r, n):
    say(f"kv append prefill r={r} n={n}")
    cfg = W.custom_config(hq=8, hkv=2, pre_chunks=((r, n),), dec_batch=3, dec_len_lo=1,
                          dec_len_hi=60, seed=r + n)
    wl = W.make_workload(cfg)
    dw = DeviceWorkload(wl)
    try:
        k_new, v_new = wl.pre_new_kv(r, n)
        # clear the new tokens' slots on the device, then append them
        for t in range(r, r + n):
            page, slot = wl.pre_bt[t // 16], t % 16
            dw.k_pool[page, :, slot] = 0
            dw.v_pool[page, :, slot] = 0
        dk, dv = _dev16(k_new, dw.device), _dev16(v_new, dw.device)
        dw.write_prefill_kv(r, n, dk, dv)
        torch.cuda.synchronize()
        assert np.array_equal(to_bits(dw.k_pool), wl.k_pool)   # incl. canary/NaN pages
        assert np.array_equal(to_bits(dw.v_pool), wl.v_pool)
    finally:
        dw.close()


def test_decode_append_and_gather_are_bit_exact():
    say("kv append decode + gather")
    cfg = W.custom_config(hq=8, hkv=2, pre_chunks=((0, 3),), dec_batch=7, dec_len_lo=1,
                          dec_len_hi=70, seed=5)
    wl = W.make_workload(cfg)
    dw = DeviceWorkload(wl)
    try:
        k_new, v_new = wl.dec_new_kv()
        for b, L in enumerate(wl.dec_lens):
            page, slot = wl.dec_bt[b, (L - 1) // 16], (L - 1) % 16
            dw.k_pool[page, :, slot] = 0
        dw.write_decode_kv(_dev16(k_new, dw.device), _dev16(v_new, dw.device))
        torch.cuda.synchronize()
        assert np.array_equal(to_bits(dw.k_pool), wl.k_pool)
        for b, L in enumerate(wl.dec_lens):
            L = int(L)
            ko = torch.empty((L, 2, 128), dtype=torch.int16, device=dw.device)
            vo = torch.empty_like(ko)
            mw.mw_kv_pool_gather(dw.pool, dw.dec_bt[b].data_ptr(), L, ko.data_ptr(), vo.data_ptr())
            k, v = wl.logical_kv(wl.dec_bt[b], L)
            torch.cuda.synchronize()
            assert np.array_equal(to_bits(ko), k) and np.array_equal(to_bits(vo), v)
    finally:
        dw.close()
