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


def probe(stream: int, n_blocks: int, spin: int, out=None, timing=None) -> torch.Tensor:
    if out is None:
        out = torch.zeros(4 * n_blocks, dtype=torch.int32, device="cuda:0")
        torch.cuda.synchronize()
    mw.mw_cu_probe(n_blocks, spin, out.data_ptr(), stream, timing)
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


def _ticks_window(raw: np.ndarray, ref: int):
    """(first start, last end) of a probe launch in 100 MHz ticks relative to
    the stamp `ref` (the stamps are the counter's low 32 bits, so differences
    are taken modulo 2^32 as signed values)."""
    def rel(x):
        return ((x.astype(np.int64) - ref + (1 << 31)) % (1 << 32)) - (1 << 31)
    return int(rel(raw[:, 2]).min()), int(rel(raw[:, 3]).max())


def test_timing_windows_agree_with_the_probe_clock():
    """The per-call timing layer against a clock inside the kernels: two probe
    launches on the two partitions (decode first), each with a timing handle.
    The event windows from mw_timing_offsets must contain the probes' own
    s_memrealtime windows and differ from them only by launch latency, the
    launch gap between the streams must be the same on both clocks, the two
    windows must overlap, and a call's elapsed time must equal the sum of its
    kernels' times."""
    from paper_2504_14489_amd.device import Timing
    say("timing windows vs probe clock")
    part = Partition(128, 128)
    d = torch.zeros(4 * 1024, dtype=torch.int32, device="cuda:0")
    p = torch.zeros_like(d)
    ta, tb = Timing(), Timing()
    torch.cuda.synchronize()
    try:
        probe(part.decode_stream, 1024, 4_000_000, d, ta.h)
        probe(part.prefill_stream, 1024, 2_000_000, p, tb.h)
        torch.cuda.synchronize()
        rd = d.cpu().numpy().astype(np.uint32).reshape(-1, 4)
        rp = p.cpu().numpy().astype(np.uint32).reshape(-1, 4)
        a0, a1 = mw.mw_timing_offsets(ta.h, ta.h)
        b0, b1 = mw.mw_timing_offsets(tb.h, ta.h)
        ea, eb = ta.elapsed()[0], tb.elapsed()[0]
        ka, kb = ta.kernel_ms(0), tb.kernel_ms(0)
    finally:
        part.close()
        ta.close()
        tb.close()
    ref = int(rd[0, 2])
    first = _ticks_window(rd, ref)[0]
    ra0, ra1 = ((x - first) / 1e5 for x in _ticks_window(rd, ref))  # ms after the decode probe's first wave
    rb0, rb1 = ((x - first) / 1e5 for x in _ticks_window(rp, ref))
    say(f"  events (ms): decode [{a0:.4f}, {a1:.4f}] prefill [{b0:.4f}, {b1:.4f}]")
    say(f"  probe clock (ms): decode [{ra0:.4f}, {ra1:.4f}] prefill [{rb0:.4f}, {rb1:.4f}]")
    tol = 0.015  # launch and event latency, ms (measured: 1-4 us)
    assert a0 == 0.0 and abs(a1 - ea) < 1e-6 and abs(b1 - b0 - eb) < 1e-3
    # each event window holds its kernel and exceeds it by launch latency only
    for (e0, e1), (r0, r1) in (((a0, a1), (ra0, ra1)), ((b0, b1), (rb0, rb1))):
        assert (r1 - r0) <= (e1 - e0) + 0.002, "event window shorter than the kernel's own"
        assert (e1 - e0) - (r1 - r0) <= tol, "event window far longer than the kernel's own"
    # the launch gap between the two streams is the same on both clocks
    assert abs((b0 - a0) - (rb0 - ra0)) <= tol
    assert abs((b1 - a0) - (rb1 - ra0)) <= tol
    # the two partitions' windows overlap, on both clocks
    assert b0 < a1 and a0 < b1 and rb0 < ra1 and ra0 < rb1
    # one kernel per call: its elapsed time is that kernel's time
    assert abs(ea - ka) < 1e-6 and abs(eb - kb) < 1e-6
