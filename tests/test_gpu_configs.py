"""Every workload at its full size on the GPU, against the oracle over whole
calls: every decode sequence of every workload, every prefill row of every
chunk (for the 8K-token long-context chunk, 512 rows covering each query block
at its tile edges, since its 2 TFLOP would take the host minutes), plus
properties that hold at any size (every output finite; multiplexed equals
isolated bit for bit).  Max-abs and mean-abs errors are taken over each
call's compared elements."""
import numpy as np
import pytest
import torch

import oracle
from paper_2504_14489_amd import workloads as W
from paper_2504_14489_amd.device import DeviceWorkload, Partition, to_bits
from tests.helpers import assert_close, say

pytestmark = pytest.mark.gpu

# workloads whose prefill chunks the oracle checks row by row in full
FULL_ROWS = {"llama8b", "llama70b", "llama70b_tp8", "sweep8b"}
NAMES = ["llama8b", "llama70b", "llama70b_tp8", "longctx8b", "sweep8b"]


def stratified_rows(n: int) -> list:
    """Rows of every 64-position query block at the edges of its 16-row
    groups (offsets 0, 15, 16, 31, 32, 47, 48, 63): both 32-position halves a
    wave owns, the first and last query of each, and the page-sized steps of
    the causal diagonal.  512 rows for a 4096-token chunk."""
    offs = (0, 15, 16, 31, 32, 47, 48, 63)
    return sorted({b + o for b in range(0, n, 64) for o in offs if b + o < n} | {n - 1})


_RUN = {}


def run_workload(name):
    """Generates the workload, runs it isolated and multiplexed on its first CU
    split and keeps the outputs (one workload held at a time)."""
    if name in _RUN:
        return _RUN[name]
    _RUN.clear()
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
        dw.o_pre.zero_()
        dw.o_dec.zero_()
        torch.cuda.synchronize()
        dw.decode(part.decode_stream)              # decode first, then prefill
        for r, n in cfg.pre_chunks:
            dw.prefill(r, n, part.prefill_stream)
        torch.cuda.synchronize()
        got_pre, got_dec = to_bits(dw.o_pre), to_bits(dw.o_dec)
    finally:
        part.close()
        dw.close()
    same = np.array_equal(iso_pre, got_pre) and np.array_equal(iso_dec, got_dec)
    _RUN[name] = (wl, got_pre, got_dec, same)
    return _RUN[name]


CASES = []
for _name in NAMES:
    CASES.append((_name, "mux"))
    CASES += [(_name, f"prefill{c}") for c in range(len(W.CONFIGS[_name].pre_chunks))]
    CASES.append((_name, "decode"))


@pytest.mark.parametrize("name,what", CASES, ids=[f"{a}-{b}" for a, b in CASES])
def test_full_size_config(name, what):
    wl, got_pre, got_dec, same = run_workload(name)
    cfg = wl.cfg
    if what == "mux":
        assert same, "multiplexed outputs differ from isolated ones"
        assert np.all(np.isfinite(W.bf16_bits_to_f32(got_pre[:wl.pre_len])))
        assert np.all(np.isfinite(W.bf16_bits_to_f32(got_dec)))
    elif what == "decode":
        B = len(wl.dec_lens)
        say(f"full-size {name}: oracle on all {B} decode sequences")
        ref = oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens)
        mx, mean = assert_close(got_dec, ref, f"{name} decode")
        say(f"  decode call: max-abs {mx:.3g} mean-abs {mean:.3g} over {B} sequences")
    else:
        r, n = cfg.pre_chunks[int(what[len("prefill"):])]
        rows = list(range(n)) if name in FULL_ROWS else stratified_rows(n)
        say(f"full-size {name}: oracle on {len(rows)} of {n} rows of chunk r={r}")
        if len(rows) == n:
            ref = oracle.prefill(wl.q_pre[r:r + n], wl.k_pool, wl.v_pool, wl.pre_bt, r)
        else:
            nvis = np.asarray([r + i + 1 for i in rows], dtype=np.int32)
            ref = oracle.paged_attention(wl.q_pre[[r + i for i in rows]], wl.k_pool, wl.v_pool,
                                         wl.pre_bt, np.zeros(len(rows), np.int32), nvis)
        mx, mean = assert_close(got_pre[[r + i for i in rows]], ref, f"{name} prefill r={r}")
        say(f"  prefill call r={r}: max-abs {mx:.3g} mean-abs {mean:.3g} over {len(rows)} rows")


def test_stratified_rows_cover_every_block_edge():
    rows = stratified_rows(4096)
    assert len(rows) == 512 and rows[0] == 0 and rows[-1] == 4095
    assert {r // 64 for r in rows} == set(range(64))


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
