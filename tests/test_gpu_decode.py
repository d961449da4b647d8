"""Decode attention on the GPU against the CPU oracle (same seeded inputs)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2504_14489_amd import workloads as W
from paper_2504_14489_amd.device import DeviceWorkload, to_bits
from tests.helpers import assert_close, say

pytestmark = pytest.mark.gpu

# lengths on and around page and chunk boundaries (16-token pages, 32-page chunks)
EDGE_LENS = [1, 2, 15, 16, 17, 31, 32, 33, 63, 64, 65, 255, 256, 257, 511, 512, 513, 1000,
             1023, 1024, 1025, 4097]


def run_decode(wl, chunk_pages=0, q_scale=None):
    dw = DeviceWorkload(wl)
    try:
        o = dw.decode(chunk_pages=chunk_pages)
        torch.cuda.synchronize()
        return to_bits(o)
    finally:
        dw.close()


@pytest.mark.parametrize("hq,hkv", [(8, 2), (32, 8), (64, 8), (4, 4), (16, 1), (6, 2)])
@pytest.mark.parametrize("q_scale", [1.0, 4.0])
def test_decode_matches_oracle_on_edge_lengths(hq, hkv, q_scale):
    say(f"decode hq={hq} hkv={hkv} q_scale={q_scale}")
    cfg = W.custom_config(hq=hq, hkv=hkv, pre_chunks=((0, 1),), dec_batch=len(EDGE_LENS),
                          seed=hq + hkv)
    wl = W.make_workload(cfg, q_scale=q_scale, dec_lens=EDGE_LENS)
    got = run_decode(wl)
    ref = oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens)
    assert_close(got, ref, f"decode hq={hq} hkv={hkv}")


@pytest.mark.parametrize("chunk_pages", [8, 16, 32, 64, -1])
def test_decode_split_count_invariance(chunk_pages):
    say(f"decode chunk_pages={chunk_pages}")
    cfg = W.custom_config(hq=32, hkv=8, pre_chunks=((0, 1),), dec_batch=12, dec_len_lo=1,
                          dec_len_hi=3000, seed=21)
    wl = W.make_workload(cfg)
    got = run_decode(wl, chunk_pages)
    ref = oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens)
    assert_close(got, ref, f"decode chunk_pages={chunk_pages}")


def test_decode_tiny_config_full_parity():
    say("decode tiny config")
    wl = W.make_workload(W.CONFIGS["tiny"])
    got = run_decode(wl)
    ref = oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens)
    assert_close(got, ref, "decode tiny")


def test_decode_page_permutation_invariance_and_determinism():
    say("decode permutation invariance")
    cfg = W.custom_config(hq=8, hkv=2, pre_chunks=((0, 1),), dec_batch=9, dec_len_lo=1,
                          dec_len_hi=900, seed=33)
    wl = W.make_workload(cfg)
    a = run_decode(wl)
    b = run_decode(wl)
    assert np.array_equal(a, b), "run-to-run results differ"
    rng = np.random.default_rng(4)
    new_of_old = rng.permutation(wl.num_pages).astype(np.int32)
    k = np.empty_like(wl.k_pool); k[new_of_old] = wl.k_pool
    v = np.empty_like(wl.v_pool); v[new_of_old] = wl.v_pool
    wl2 = W.Workload(cfg=wl.cfg, k_pool=k, v_pool=v, nan_page=int(new_of_old[wl.nan_page]),
                     pre_len=wl.pre_len, pre_bt=new_of_old[wl.pre_bt], q_pre=wl.q_pre,
                     dec_lens=wl.dec_lens, dec_bt=new_of_old[wl.dec_bt], q_dec=wl.q_dec,
                     perm=wl.perm)
    c = run_decode(wl2)
    assert np.array_equal(a, c), "page renumbering changed the result"


def test_decode_equals_last_prefill_row():
    say("decode vs last prefill row")
    from paper_2504_14489_amd.device import DeviceWorkload as DW
    cfg = W.custom_config(hq=8, hkv=2, pre_chunks=((0, 77),), dec_batch=1, dec_len_lo=1,
                          dec_len_hi=2, seed=8)
    wl = W.make_workload(cfg)
    dw = DW(wl)
    try:
        pre = to_bits(dw.prefill(0, 77))[-1]
        # decode the last prefill token over the same 77-token sequence
        dw.q_dec = dw.q_pre[76:77].contiguous()
        dw.dec_bt = dw.pre_bt
        dw.dec_lens = np.array([77], np.int32)
        dw.d_dec_lens = torch.tensor([77], dtype=torch.int32, device=dw.device)
        dw.o_dec = torch.zeros_like(dw.q_dec)
        dw._ws.clear()
        dec = to_bits(dw.decode())[0]
        torch.cuda.synchronize()
    finally:
        dw.close()
    ref = oracle.prefill(wl.q_pre[76:77], wl.k_pool, wl.v_pool, wl.pre_bt, 76)[0]
    assert_close(pre[None], ref[None], "prefill last row")
    assert_close(dec[None], ref[None], "decode")
    diff = np.abs(W.bf16_bits_to_f32(pre) - W.bf16_bits_to_f32(dec))
    assert diff.max() <= 2e-2


def test_decode_wide_score_range():
    """Keys scaled by 32 against Q scaled by 8, placed in different chunks and
    in both halves of an 8-key group: the split maxima and the combine must
    keep every 2^(s - m) finite."""
    say("decode wide score range")
    from paper_2504_14489_amd.device import bits_to_f32
    cfg = W.custom_config(hq=8, hkv=2, pre_chunks=((0, 1),), dec_batch=3, seed=78)
    wl = W.make_workload(cfg, q_scale=8.0, dec_lens=[700, 1500, 33])
    k = wl.k_pool.copy()
    for b, positions in enumerate([[5, 500, 699], [6, 600, 1200, 1499], [1, 32]]):
        for t in positions:
            page, slot = wl.dec_bt[b, t // 16], t % 16
            row = bits_to_f32(k[page, :, slot, :]) * 32.0
            k[page, :, slot, :] = (row.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    wl = W.Workload(cfg=wl.cfg, k_pool=k, v_pool=wl.v_pool, nan_page=wl.nan_page, pre_len=wl.pre_len,
                    pre_bt=wl.pre_bt, q_pre=wl.q_pre, dec_lens=wl.dec_lens, dec_bt=wl.dec_bt,
                    q_dec=wl.q_dec, perm=wl.perm)
    got = run_decode(wl)
    ref = oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens)
    assert_close(got, ref, "decode wide score range")


# (name, hq, hkv, batch, shortest, longest): long sequences whose segments the
# balanced ranges cut, and many 1..3-page sequences several of whose segments
# fall in one range; then few long sequences, whose segments the split pads to
# a multiple of the range (one sequence of 139 pages, a prime; one of 34 pages,
# cut 16 + 16 + 2; three of unequal lengths)
BALANCED_CASES = [("long", 32, 8, 24, 1, 3000), ("short", 8, 2, 300, 1, 40), ("group16", 16, 1, 5, 700, 4100),
                  ("one139", 32, 8, 1, 2213, 2213), ("one34", 32, 8, 1, 530, 530),
                  ("three", 32, 8, 3, 9000, 20000)]


@pytest.mark.parametrize("decode_cus", [8, 64, 192, 256])
@pytest.mark.parametrize("case", BALANCED_CASES, ids=[c[0] for c in BALANCED_CASES])
def test_decode_balanced_split_on_partitions(case, decode_cus):
    """The balanced split (chunk_pages 0) cuts the pages into 2 ranges per CU
    of the stream: every partition size gives the oracle's result, run to run
    bit for bit, and the same bits as a second stream of that size."""
    from paper_2504_14489_amd.device import Partition
    name, hq, hkv, batch, lo, hi = case
    say(f"decode balanced {name} on {decode_cus} CUs")
    cfg = W.custom_config(hq=hq, hkv=hkv, pre_chunks=((0, 1),), dec_batch=batch, dec_len_lo=lo,
                          dec_len_hi=hi, seed=50 + batch)
    wl = W.make_workload(cfg)
    dw = DeviceWorkload(wl)
    parts = []
    try:
        if decode_cus < 256:
            parts = [Partition(256 - decode_cus, decode_cus), Partition(256 - decode_cus, decode_cus)]
            streams = [p.decode_stream for p in parts]
        else:
            streams = [0, torch.cuda.Stream().cuda_stream]
        outs = []
        for st in streams + streams[:1]:
            o = dw.decode(st)
            torch.cuda.synchronize()
            outs.append(to_bits(o))
    finally:
        for p in parts:
            p.close()
        dw.close()
    assert np.array_equal(outs[0], outs[2]), "run-to-run results differ"
    assert np.array_equal(outs[0], outs[1]), "two streams of one size differ"
    ref = oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens)
    assert_close(outs[0], ref, f"decode balanced {name} on {decode_cus} CUs")



@pytest.mark.parametrize("slack", [(W.BF16_NAN, W.BF16_NAN), (W.BF16_POS_INF, W.BF16_NEG_INF)],
                         ids=["nan-nan", "inf-neginf"])
@pytest.mark.parametrize("chunk_pages", [0, 8])
def test_decode_ignores_nan_and_inf_in_slack_slots(slack, chunk_pages):
    """Slots past each sequence's end in its last page hold NaN or Inf: the
    keys there are masked and their values must never reach the output (the
    balanced split and fixed chunks; lengths on and around page edges)."""
    say(f"decode slack {slack} chunk_pages={chunk_pages}")
    cfg = W.custom_config(hq=32, hkv=8, pre_chunks=((0, 1),), dec_batch=len(EDGE_LENS), seed=5)
    wl = W.make_workload(cfg, dec_lens=EDGE_LENS, slack_bits=slack)
    got = run_decode(wl, chunk_pages)
    ref = oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens)
    assert_close(got, ref, f"decode slack chunk_pages={chunk_pages}")


def test_decode_segment_flags_with_any_workspace_contents():
    """The balanced split merges each (sequence, kv head) in the work-group
    that finds all of its pieces done, through per-piece flags in the
    workspace: the result must not depend on what the workspace held before
    (never written, all ones, random bytes, an earlier call's flags)."""
    say("decode segment flags: workspace contents")
    cfg = W.custom_config(hq=32, hkv=8, pre_chunks=((0, 1),), dec_batch=5, dec_len_lo=2000,
                          dec_len_hi=9000, seed=51)
    wl = W.make_workload(cfg)
    ref = oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens)
    dw = DeviceWorkload(wl)
    try:
        ws = dw.workspace(0)
        gen = torch.Generator(device=dw.device).manual_seed(3)
        results = []
        for fill in ("as allocated", "ones", "random", "reused", "reused"):
            if fill == "ones":
                ws.fill_(255)
            elif fill == "random":
                ws.copy_(torch.randint(0, 256, ws.shape, generator=gen, device=dw.device, dtype=torch.uint8))
            dw.o_dec.zero_()
            got = to_bits(dw.decode())
            torch.cuda.synchronize()
            assert_close(got, ref, f"decode, workspace {fill}")
            results.append(got)
        for got in results[1:]:
            assert np.array_equal(got, results[0]), "the result depends on the workspace contents"
    finally:
        dw.close()


def test_decode_one_segment_in_hundreds_of_pieces():
    """One sequence, one kv head: the whole call is a single segment cut into
    as many pieces as the split has units (hundreds of flags per merge)."""
    say("decode one segment, many pieces")
    cfg = W.custom_config(hq=16, hkv=1, pre_chunks=((0, 1),), dec_batch=1, dec_len_lo=70001,
                          dec_len_hi=70002, seed=52)
    wl = W.make_workload(cfg)
    ref = oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens)
    dw = DeviceWorkload(wl)
    try:
        for rep in range(3):
            dw.o_dec.zero_()
            got = to_bits(dw.decode())
            torch.cuda.synchronize()
            assert_close(got, ref, f"decode one segment, call {rep}")
    finally:
        dw.close()


def test_decode_random_batches_on_partitions():
    """Random small batches (1-6 sequences of 1..20000 tokens, equal or not)
    with random head shapes on random partition sizes: whichever balanced
    split the planner takes (ranges across segments, or segments padded to
    whole ranges), the result is the oracle's."""
    from paper_2504_14489_amd.device import Partition
    rng = np.random.default_rng(77)
    for case in range(12):
        hkv = int(rng.choice([1, 2, 8]))
        hq = hkv * int(rng.choice([1, 4, 8]))
        batch = int(rng.integers(1, 7))
        if case % 3 == 0:
            lens = [int(rng.integers(1, 20001))] * batch
        else:
            lens = [int(x) for x in rng.integers(1, 20001, batch)]
        decode_cus = int(rng.choice([8, 32, 96, 160, 256]))
        say(f"decode random case {case}: hq={hq} hkv={hkv} lens={lens} on {decode_cus} CUs")
        cfg = W.custom_config(hq=hq, hkv=hkv, pre_chunks=((0, 1),), dec_batch=batch, seed=200 + case)
        wl = W.make_workload(cfg, dec_lens=lens)
        dw = DeviceWorkload(wl)
        part = None
        try:
            if decode_cus < 256:
                part = Partition(256 - decode_cus, decode_cus)
                stream = part.decode_stream
            else:
                stream = 0
            got = to_bits(dw.decode(stream))
            torch.cuda.synchronize()
        finally:
            if part is not None:
                part.close()
            dw.close()
        ref = oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens)
        assert_close(got, ref, f"decode random case {case}")


def test_decode_graph_replays_reuse_the_tag():
    """A decode call captured in a graph replays with the tag it was captured
    with: the merging work-group clears the segment's flags, so every replay
    merges again, also with eager calls (other tags) on the same workspace
    in between.  One 20,001-token sequence on the whole GPU: a split whose
    segments are padded to whole ranges."""
    say("decode graph replays")
    cfg = W.custom_config(hq=32, hkv=8, pre_chunks=((0, 1),), dec_batch=1, seed=91)
    wl = W.make_workload(cfg, dec_lens=[20001])
    dw = DeviceWorkload(wl)
    try:
        ref = to_bits(dw.decode()).copy()
        torch.cuda.synchronize()
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            dw.decode(s.cuda_stream)  # warm-up on the capture stream
        s.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            dw.decode(torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        other = torch.empty_like(dw.o_dec)
        for rep in range(4):
            dw.o_dec.zero_()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert np.array_equal(to_bits(dw.o_dec), ref), f"replay {rep}"
            dw.decode(out=other)  # an eager call with its own tag, same workspace
            torch.cuda.synchronize()
            assert np.array_equal(to_bits(other), ref), f"eager call after replay {rep}"
        del g
    finally:
        dw.close()
    assert_close(ref, oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens), "decode graph case")
