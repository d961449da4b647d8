"""The multiplex engine's host loop (paper Sec. 3.2): blocking and polled
coordination, layer-wise prefill launches and the switch to the whole device
must leave every output identical to one plain call, and its timeline
statistics must describe what ran."""
import numpy as np
import pytest
import torch

from paper_2504_14489_amd import mw, workloads as W
from paper_2504_14489_amd.device import DeviceWorkload, to_bits
from paper_2504_14489_amd.engine import Engine
import oracle
from tests.helpers import assert_close, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def setup():
    cfg = W.custom_config("engine", hq=8, hkv=2, pre_chunks=((0, 200), (200, 180)), dec_batch=6,
                          dec_len_lo=100, dec_len_hi=900)
    wl = W.make_workload(cfg, seed=11)
    dw = DeviceWorkload(wl)
    eng = Engine([64, 128])
    dec, pre = dw.engine_args()
    yield wl, dw, eng, dec, pre
    eng.close()
    dw.close()


def _plain_outputs(dw, eng, dec, pre, config=-1):
    """One decode and one prefill call on the streams of partition `config`
    (-1: the whole device).  The decode split depends on the stream's CU
    count, so a run on a partition is compared with a call on its stream."""
    ps, ds = eng.streams(config)
    mw.mw_decode_attn(dec["pool"], dw.hq, dw.hkv, dw.d, dw.scale, dw.dec_lens, dec["d_seq_lens"],
                      dec["d_block_table"], dec["bt_stride"], dec["d_q"], dec["d_out"], dec["d_workspace"],
                      dec["workspace_bytes"], 0, ds, None)
    mw.mw_prefill_attn(pre["pool"], dw.hq, dw.hkv, dw.d, dw.scale, pre["new_lens"], pre["prefix_lens"],
                       pre["d_qo_indptr"], pre["d_prefix_lens"], pre["d_block_table"], pre["bt_stride"],
                       pre["d_q"], pre["d_out"], ps, None)
    mw.mw_sync(ps)
    mw.mw_sync(ds)
    return dw.o_dec.clone(), dw.o_pre.clone()


def test_engine_batch_of_chunks_matches_oracle(setup):
    """The prefill batch the engine runs (every chunk in one call) and the
    decode call agree with the oracle."""
    wl, dw, eng, dec, pre = setup
    say("engine: plain outputs vs oracle")
    o_dec, o_pre = _plain_outputs(dw, eng, dec, pre)
    c = wl.cfg
    ref_pre = oracle.prefill(wl.q_pre[:c.pre_total], wl.k_pool, wl.v_pool, wl.pre_bt, 0)
    assert_close(to_bits(o_pre[:c.pre_total]), ref_pre, "engine prefill batch")
    ref_dec = oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens)
    assert_close(to_bits(o_dec), ref_dec, "engine decode")


@pytest.mark.parametrize("policy,npl,switch", [
    (mw.MW_ENGINE_BLOCKING, 24, False),
    (mw.MW_ENGINE_POLLED, 3, False),
    (mw.MW_ENGINE_POLLED, 3, True),
    (mw.MW_ENGINE_POLLED, 1, True),
])
@pytest.mark.parametrize("config", [0, 1])
def test_engine_runs_leave_outputs_unchanged(setup, policy, npl, switch, config):
    wl, dw, eng, dec, pre = setup
    say(f"engine run: policy {policy} N_PL {npl} switch {switch} partition {config}")
    ref_dec, ref_pre = _plain_outputs(dw, eng, dec, pre, config)
    dw.o_dec.zero_()
    dw.o_pre.zero_()
    torch.cuda.synchronize()
    iters, layers, pl = 3, 4, 24
    s = eng.run(dec, pre, config=config, decode_iters=iters, decode_layers=layers, prefill_layers=pl,
                layers_per_launch=npl, policy=policy, switch_on_decode_end=switch)
    assert torch.equal(dw.o_dec, ref_dec) and torch.equal(dw.o_pre, ref_pre)
    td, tpf = mw.mw_engine_timeline(eng.h, 0), mw.mw_engine_timeline(eng.h, 1)
    assert td.shape == (iters * layers, 3) and tpf.shape == (pl, 3)
    for tl in (td, tpf):                 # calls of one stream: in order, no overlap
        assert np.all(tl[:, 1] >= tl[:, 0]) and np.all(tl[1:, 0] >= tl[:-1, 1] - 1e-3)
    assert abs((td[:, 1] - td[:, 0]).sum() - s["decode_busy_ms"]) < 1e-3
    assert abs((tpf[:, 1] - tpf[:, 0]).sum() - s["prefill_busy_ms"]) < 1e-3
    assert int(tpf[:, 2].sum()) == s["switched_layers"]
    assert 0.0 <= s["decode_bubble"] < 1.0 and 0.0 <= s["prefill_bubble"] < 1.0
    assert s["bubble_ratio"] == pytest.approx(0.5 * (s["decode_bubble"] + s["prefill_bubble"]))
    assert 0.0 < s["decode_busy_ms"] <= s["wall_ms"] + 1e-6
    assert 0.0 < s["prefill_busy_ms"] <= s["wall_ms"] + 1e-6
    assert s["prefill_end_ms"] <= s["wall_ms"] + 1e-6
    assert s["decode_iter_ms_mean"] > 0.0 and s["decode_gap_ms_max"] >= 0.0
    if policy == mw.MW_ENGINE_BLOCKING:
        assert s["prefill_batches"] == 1 and s["switched_layers"] == 0
    else:
        assert s["prefill_batches"] >= -(-pl // npl)
        assert 0 <= s["switched_layers"] <= pl
        if not switch:
            assert s["switched_layers"] == 0 and s["switch_gap_ms"] == -1.0
        elif s["switched_layers"] > 0:
            assert s["switch_host_us"] >= 0.0


def test_engine_switch_moves_late_layers_to_the_whole_device(setup):
    """One short decode iteration and a long prefill: with N_PL = 1 almost
    every prefill layer is still unlaunched when decode ends, so they move."""
    wl, dw, eng, dec, pre = setup
    say("engine switch")
    s = eng.run(dec, pre, config=0, decode_iters=1, decode_layers=1, prefill_layers=64,
                layers_per_launch=1, policy=mw.MW_ENGINE_POLLED, switch_on_decode_end=True)
    assert s["switched_layers"] > 0
    assert s["switch_gap_ms"] >= 0.0 and s["switch_host_us"] >= 0.0
    assert s["prefill_batches"] == 64


def test_engine_group_memory_and_streams(setup):
    wl, dw, eng, dec, pre = setup
    nbytes, ms = eng.memory()
    assert ms > 0.0 and nbytes >= 0
    p0, d0 = eng.streams(0)
    p1, d1 = eng.streams(1)
    pw, dwh = eng.streams(-1)
    assert len({p0, d0, p1, d1}) == 4 and pw == dwh
    with pytest.raises(mw.MWError):
        eng.streams(2)
    with pytest.raises(mw.MWError):
        eng.run(dec, pre, config=2, decode_iters=1, decode_layers=1, prefill_layers=1, layers_per_launch=1)
    with pytest.raises(mw.MWError):
        eng.run(dec, pre, config=0, decode_iters=0, decode_layers=1, prefill_layers=1, layers_per_launch=1)


def test_engine_rejects_bad_partitions():
    for cus in ([0], [60], [256], [-8]):
        with pytest.raises(mw.MWError):
            Engine(cus)


def test_engine_decode_graph_replays_match_eager(setup):
    """Decode iterations as graph launches: every replay recomputes the
    outputs (zeroed before each run, eager calls in between) and one graph
    serves every run with the same arguments and partition."""
    wl, dw, eng, dec, pre = setup
    say("engine decode graph replays")
    ref_dec, ref_pre = _plain_outputs(dw, eng, dec, pre, 0)
    n0 = eng.graphs()[0]
    for rep in range(4):
        dw.o_dec.zero_()
        dw.o_pre.zero_()
        torch.cuda.synchronize()
        s = eng.run(dec, pre, config=0, decode_iters=3, decode_layers=4, prefill_layers=12,
                    layers_per_launch=3, policy=mw.MW_ENGINE_POLLED, switch_on_decode_end=True,
                    decode_graph=True)
        assert torch.equal(dw.o_dec, ref_dec), f"replay {rep}"
        assert torch.equal(dw.o_pre, ref_pre), f"replay {rep}"
        assert mw.mw_engine_timeline(eng.h, 0).shape == (3, 3)      # one span per iteration
        assert s["decode_iter_ms_mean"] > 0.0
        _plain_outputs(dw, eng, dec, pre, 0)                         # eager work between replays
    n1, nbytes, ms = eng.graphs()
    assert n1 == n0 + 1 and nbytes >= 0 and ms > 0.0
    eng.run(dec, pre, config=1, decode_iters=1, decode_layers=4, prefill_layers=2, layers_per_launch=1,
            decode_graph=True)
    eng.run(dec, pre, config=0, decode_iters=1, decode_layers=2, prefill_layers=2, layers_per_launch=1,
            decode_graph=True)
    assert eng.graphs()[0] == n0 + 3                                  # per partition and layer count
    assert torch.equal(dw.o_dec, ref_dec)


def test_graph_launched_on_a_partition_stream_keeps_its_cus():
    """A graph replayed on a CU-masked stream runs its kernels on that
    stream's CUs only (what per-partition decode graphs rely on)."""
    from paper_2504_14489_amd.device import Partition
    from tests.test_gpu_partition import cu_ids
    say("graph on a masked stream")
    part = Partition(64, 192)
    n_blocks = 2048
    eager = torch.zeros(4 * n_blocks, dtype=torch.int32, device="cuda:0")
    graphed = torch.zeros_like(eager)
    torch.cuda.synchronize()
    try:
        mw.mw_cu_probe(n_blocks, 20000, eager.data_ptr(), part.decode_stream)
        mw.mw_sync(part.decode_stream)
        ext = torch.cuda.ExternalStream(part.decode_stream)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=ext):
            mw.mw_cu_probe(n_blocks, 20000, graphed.data_ptr(), part.decode_stream)
        for _ in range(2):
            graphed.zero_()
            torch.cuda.synchronize()
            with torch.cuda.stream(ext):
                g.replay()
            torch.cuda.synchronize()
            got = {tuple(x) for x in cu_ids(graphed.cpu().numpy().astype(np.uint32).reshape(-1, 4))}
            want = {tuple(x) for x in cu_ids(eager.cpu().numpy().astype(np.uint32).reshape(-1, 4))}
            assert len(want) == 192 and got <= want, f"{len(got - want)} CUs outside the partition"
        del g
    finally:
        part.close()


def test_engine_prefill_with_split_workspace():
    """Prefill arguments that carry a workspace make the engine issue
    key-range-split calls: a short chunk over a long prefix with one kv head
    has too few query blocks for a 64-CU partition, so the call is cut; the
    engine's outputs equal one split call on that partition's stream, and
    the oracle's."""
    from paper_2504_14489_amd.device import Timing
    cfg = W.custom_config("engine_split", hq=8, hkv=1, pre_chunks=((2000, 64),), dec_batch=3,
                          dec_len_lo=100, dec_len_hi=400)
    wl = W.make_workload(cfg, seed=12)
    dw = DeviceWorkload(wl)
    eng = Engine([64])
    try:
        dec, pre = dw.engine_args()
        nbytes = mw.mw_prefill_workspace_size(dw.hq, dw.hkv, dw.d, pre["new_lens"], pre["prefix_lens"], 64)
        assert nbytes > 0, "the plan does not cut on 64 CUs"
        ws = torch.empty(nbytes, dtype=torch.uint8, device=dw.device)
        pre = dict(pre, d_workspace=ws.data_ptr(), workspace_bytes=ws.numel())
        say("engine run with a split prefill workspace")
        ps, ds = eng.streams(0)
        t = Timing()
        mw.mw_prefill_attn_ws(pre["pool"], dw.hq, dw.hkv, dw.d, dw.scale, pre["new_lens"], pre["prefix_lens"],
                              pre["d_qo_indptr"], pre["d_prefix_lens"], pre["d_block_table"], pre["bt_stride"],
                              pre["d_q"], pre["d_out"], ws.data_ptr(), ws.numel(), ps, t.h)
        mw.mw_sync(ps)
        assert t.kernels() == 2, "the plain split call did not cut"
        ref_pre = dw.o_pre.clone()
        dw.o_pre.zero_()
        torch.cuda.synchronize()
        eng.run(dec, pre, config=0, decode_iters=2, decode_layers=2, prefill_layers=6, layers_per_launch=2,
                policy=mw.MW_ENGINE_POLLED, switch_on_decode_end=False)
        assert torch.equal(dw.o_pre, ref_pre), "engine prefill differs from the split call"
        c = wl.cfg
        ref = oracle.prefill(wl.q_pre[2000:2064], wl.k_pool, wl.v_pool, wl.pre_bt, 2000)
        assert_close(to_bits(dw.o_pre[2000:2064]), ref, "engine split prefill")
    finally:
        eng.close()
        dw.close()
