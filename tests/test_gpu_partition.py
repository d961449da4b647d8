"""CU-masked partitions: the probe kernel reads the hardware ids of the CU each
work-group runs on, so the masks' meaning is checked on the device itself."""
import numpy as np
import pytest
import torch

from paper_2504_14489_amd import mw
from paper_2504_14489_amd.device import Partition
from tests.helpers import say

pytestmark = pytest.mark.gpu


def cu_ids(raw: np.ndarray):
    """(xcc, se, sh, cu) per work-group from the probe's XCC_ID and HW_ID words."""
    xcc = raw[:, 0] & 0xF
    hw = raw[:, 1]
    return np.stack([xcc, (hw >> 13) & 0x7, (hw >> 12) & 0x1, (hw >> 8) & 0xF], axis=1)


def probe(stream: int, n_blocks: int, spin: int, out=None) -> torch.Tensor:
    if out is None:
        out = torch.zeros(4 * n_blocks, dtype=torch.int32, device="cuda:0")
        torch.cuda.synchronize()
    mw.mw_cu_probe(n_blocks, spin, out.data_ptr(), stream)
    return out


@pytest.mark.parametrize("p_cus,d_cus", [(64, 192), (128, 128), (32, 224), (96, 160)])
def test_partition_masks_select_disjoint_cus_evenly_over_xcds(p_cus, d_cus):
    say(f"partition probe {p_cus}/{d_cus}")
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    part = Partition(p_cus, d_cus)
    try:
        a = probe(part.prefill_stream, 4096, 20000)
        b = probe(part.decode_stream, 4096, 20000)
        torch.cuda.synchronize()
        ia = cu_ids(a.cpu().numpy().astype(np.uint32).reshape(-1, 4))
        ib = cu_ids(b.cpu().numpy().astype(np.uint32).reshape(-1, 4))
    finally:
        part.close()
    sa = {tuple(x) for x in ia}
    sb = {tuple(x) for x in ib}
    say(f"  distinct CUs: prefill {len(sa)} decode {len(sb)} of {n_cu}")
    assert not (sa & sb), "a CU ran work of both partitions"
    assert len(sa) == p_cus and len(sb) == d_cus
    n_xcc = len({x[0] for x in sa | sb})
    for s, want in ((sa, p_cus), (sb, d_cus)):
        per = np.bincount([x[0] for x in s], minlength=n_xcc)
        assert np.all(per == want // n_xcc), f"uneven CUs per XCD: {per}"


def test_partition_streams_run_concurrently():
    say("partition concurrency")
    part = Partition(128, 128)
    # buffers first: work on the null stream would serialise with both
    # (blocking) partition streams
    d = torch.zeros(4 * 8192, dtype=torch.int32, device="cuda:0")
    p = torch.zeros_like(d)
    torch.cuda.synchronize()
    try:
        probe(part.decode_stream, 8192, 400000, d)
        probe(part.prefill_stream, 8192, 400000, p)
        torch.cuda.synchronize()
        rd = d.cpu().numpy().astype(np.uint32).reshape(-1, 4).astype(np.int64)
        rp = p.cpu().numpy().astype(np.uint32).reshape(-1, 4).astype(np.int64)
    finally:
        part.close()
    base = min(rd[:, 2].min(), rp[:, 2].min())
    d0, d1 = rd[:, 2].min() - base, rd[:, 3].max() - base
    p0, p1 = rp[:, 2].min() - base, rp[:, 3].max() - base
    overlap = min(d1, p1) - max(d0, p0)
    say(f"  decode [{d0}, {d1}] prefill [{p0}, {p1}] (100 MHz ticks)")
    assert overlap > 0.5 * min(d1 - d0, p1 - p0), "the two partitions did not overlap in time"
