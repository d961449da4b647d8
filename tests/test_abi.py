"""The C ABI without a GPU: the library loads, exports every entry point that
include/mw.h declares, and its host-side logic (argument validation, the page
allocator, workspace sizing) behaves as documented.  No call here launches a
kernel."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2504_14489_amd import build as B
from paper_2504_14489_amd import mw

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_entry_points():
    text = open(os.path.join(ROOT, "include", "mw.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mw_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(mw.LIB_PATH):
        B.build()
    return mw.load()


def test_every_declared_symbol_is_exported_and_bound(lib):
    names = declared_entry_points()
    assert len(names) >= 25
    for n in names:
        assert hasattr(lib, n), f"{n} is declared in mw.h but not exported"
    assert sorted(mw.EXPORTED) == names


def test_version_and_empty_error(lib):
    assert mw.mw_version() == 2


FAKE_K, FAKE_V = 0x10000, 0x20000     # aligned addresses that are never dereferenced


def test_pool_allocator_host_logic(lib):
    pool = mw.mw_kv_pool_create(10, 16, 2, 128, FAKE_K, FAKE_V)
    try:
        assert mw.mw_kv_pool_num_free(pool) == 10
        mw.mw_kv_pool_set_free_order(pool, [7, 3, 9, 1])
        assert mw.mw_kv_pool_num_free(pool) == 4
        assert list(mw.mw_kv_pool_alloc(pool, 3)) == [7, 3, 9]
        with pytest.raises(mw.MWError) as e:
            mw.mw_kv_pool_alloc(pool, 2)
        assert e.value.status == mw.MW_ERR_OUT_OF_PAGES
        assert mw.mw_kv_pool_num_free(pool) == 1        # a failed alloc takes nothing
        mw.mw_kv_pool_free(pool, [3, 7])
        assert list(mw.mw_kv_pool_alloc(pool, 3)) == [1, 3, 7]
        for bad in ([1, 1], [10], [-1]):
            with pytest.raises(mw.MWError) as e:
                mw.mw_kv_pool_free(pool, bad) if bad != [1, 1] else mw.mw_kv_pool_set_free_order(pool, bad)
            assert e.value.status == mw.MW_ERR_INVALID_ARG
        mw.mw_kv_pool_free(pool, [9])
        with pytest.raises(mw.MWError):                  # 9 is already free
            mw.mw_kv_pool_free(pool, [9])
    finally:
        mw.mw_kv_pool_destroy(pool)


@pytest.mark.parametrize("args,status", [
    ((10, 8, 2, 128), mw.MW_ERR_UNSUPPORTED),
    ((10, 16, 2, 64), mw.MW_ERR_UNSUPPORTED),
    ((0, 16, 2, 128), mw.MW_ERR_INVALID_ARG),
    ((10, 16, 0, 128), mw.MW_ERR_INVALID_ARG),
])
def test_pool_create_validation(lib, args, status):
    with pytest.raises(mw.MWError) as e:
        mw.mw_kv_pool_create(*args, FAKE_K, FAKE_V)
    assert e.value.status == status
    with pytest.raises(mw.MWError) as e:
        mw.mw_kv_pool_create(10, 16, 2, 128, FAKE_K + 8, FAKE_V)   # misaligned
    assert e.value.status == mw.MW_ERR_INVALID_ARG
    assert "aligned" in mw.mw_last_error()


def test_decode_workspace_size(lib):
    # 3 sequences of 1, 16*16, 16*16+1 tokens with 16-page chunks: 1 + 1 + 2 chunks
    n = mw.mw_decode_workspace_size(8, 2, 128, [1, 256, 257], 16)
    units = 4 * 2
    assert n >= units * 4 * 128 * 4 + units * 4 * 8 + 3 * 4
    assert mw.mw_decode_workspace_size(8, 2, 128, [1, 256, 257], 8) > n
    for args, status in [((8, 3, 128, [5]), mw.MW_ERR_INVALID_ARG),
                         ((8, 2, 64, [5]), mw.MW_ERR_UNSUPPORTED),
                         ((64, 2, 128, [5]), mw.MW_ERR_UNSUPPORTED),
                         ((8, 2, 128, [0]), mw.MW_ERR_INVALID_ARG)]:
        with pytest.raises(mw.MWError) as e:
            mw.mw_decode_workspace_size(*args)
        assert e.value.status == status
    for bad in (4, 12, 264, -2, -8):
        with pytest.raises(mw.MWError) as e:
            mw.mw_decode_workspace_size(8, 2, 128, [5], bad)
        assert e.value.status == mw.MW_ERR_UNSUPPORTED


def test_prefill_workspace_size(lib):
    """The split's workspace: pieces x rows x q heads x (512 + 8) bytes.  With
    no CU count it covers the most pieces (8) any stream's plan can take; on a
    given CU count the plan cuts only launches of 4-wave blocks (their pairs of
    64-position blocks fewer than the CUs) and never more than that bound."""
    row_bytes = 128 * 4 + 8
    # a one-kv-head shard: 8 q heads, 2048 new tokens over 6144 cached (blocks of
    # 97..128 key tiles): 32 pairs x 2 head groups = 64 < 96 CUs -> 4-wave blocks
    assert mw.mw_prefill_workspace_size(8, 1, 128, [2048], [6144], 0) == 8 * 2048 * 8 * row_bytes
    for cus in (96, 128, 256):
        b = mw.mw_prefill_workspace_size(8, 1, 128, [2048], [6144], cus)
        assert b % (2048 * 8 * row_bytes) == 0 and 2 <= b // (2048 * 8 * row_bytes) <= 8, (cus, b)
    # 8-wave launches (enough pairs for every CU) are never cut
    assert mw.mw_prefill_workspace_size(8, 1, 128, [2048], [6144], 64) == 0
    assert mw.mw_prefill_workspace_size(64, 8, 128, [2048], [6144], 96) == 0
    # a varlen batch: rows of both sequences; the longest block decides the pieces
    assert mw.mw_prefill_workspace_size(8, 2, 128, [100, 33], [0, 4100], 0) == 8 * 133 * 8 * row_bytes
    # nothing to cut: blocks of at most 4 key tiles
    assert mw.mw_prefill_workspace_size(8, 2, 128, [200], [0], 0) == 0
    assert mw.mw_prefill_workspace_size(8, 2, 128, [], [], 0) == 0
    for args, status in [((8, 3, 128, [5], [0], 0), mw.MW_ERR_INVALID_ARG),
                         ((8, 2, 64, [5], [0], 0), mw.MW_ERR_UNSUPPORTED),
                         ((8, 2, 128, [-1], [0], 0), mw.MW_ERR_INVALID_ARG),
                         ((8, 2, 128, [5], [-3], 0), mw.MW_ERR_INVALID_ARG),
                         ((8, 2, 128, [5], [0], -1), mw.MW_ERR_INVALID_ARG)]:
        with pytest.raises(mw.MWError) as e:
            mw.mw_prefill_workspace_size(*args)
        assert e.value.status == status


def test_attention_calls_reject_bad_arguments_before_launching(lib):
    pool = mw.mw_kv_pool_create(10, 16, 2, 128, FAKE_K, FAKE_V)
    try:
        with pytest.raises(mw.MWError) as e:          # prefix + new beyond the table
            mw.mw_prefill_attn(pool, 4, 2, 128, 0.1, [20], [0], 0x100, 0x200, 0x300, 1,
                               0x400, 0x500)
        assert e.value.status == mw.MW_ERR_INVALID_ARG
        with pytest.raises(mw.MWError) as e:          # kv heads differ from the pool's
            mw.mw_prefill_attn(pool, 4, 4, 128, 0.1, [4], [0], 0x100, 0x200, 0x300, 1, 0x400,
                               0x500)
        assert e.value.status == mw.MW_ERR_INVALID_ARG
        with pytest.raises(mw.MWError) as e:          # misaligned Q
            mw.mw_prefill_attn(pool, 4, 2, 128, 0.1, [4], [0], 0x100, 0x200, 0x300, 1, 0x408,
                               0x500)
        assert e.value.status == mw.MW_ERR_INVALID_ARG
        with pytest.raises(mw.MWError) as e:          # non-positive scale
            mw.mw_prefill_attn(pool, 4, 2, 128, 0.0, [4], [0], 0x100, 0x200, 0x300, 1, 0x400,
                               0x500)
        assert e.value.status == mw.MW_ERR_INVALID_ARG
        with pytest.raises(mw.MWError) as e:          # workspace too small
            mw.mw_decode_attn(pool, 4, 2, 128, 0.1, [17], 0x100, 0x200, 2, 0x300, 0x400, 0x500,
                              16)
        assert e.value.status == mw.MW_ERR_INVALID_ARG
        with pytest.raises(mw.MWError) as e:          # length beyond the table
            mw.mw_decode_attn(pool, 4, 2, 128, 0.1, [33], 0x100, 0x200, 2, 0x300, 0x400, 0x500,
                              1 << 20)
        assert e.value.status == mw.MW_ERR_INVALID_ARG
        with pytest.raises(mw.MWError) as e:          # writes beyond the table
            mw.mw_kv_pool_write(pool, [5], [30], 0x100, 0x200, 0x300, 2, 0x400, 0x500)
        assert e.value.status == mw.MW_ERR_INVALID_ARG
    finally:
        mw.mw_kv_pool_destroy(pool)


def test_partition_validation(lib):
    for p, d in ((12, 64), (64, 0), (128, 136), (0, 8)):
        with pytest.raises(mw.MWError) as e:
            mw.mw_partition_create(0, p, d)
        assert e.value.status in (mw.MW_ERR_INVALID_ARG, mw.MW_ERR_HIP)
    with pytest.raises(mw.MWError) as e:
        mw.mw_partition_create_masks(0, [1, 0], [1, 0])
    assert e.value.status in (mw.MW_ERR_INVALID_ARG, mw.MW_ERR_HIP)


def test_timing_not_ready(lib):
    t = mw.mw_timing_create()
    try:
        with pytest.raises(mw.MWError) as e:
            mw.mw_timing_elapsed(t)
        assert e.value.status == mw.MW_ERR_NOT_READY
        assert mw.mw_timing_kernels(t) == 0
    finally:
        mw.mw_timing_destroy(t)


def test_engine_validation_without_a_device(lib):
    with pytest.raises(mw.MWError) as e:
        mw.mw_engine_create(0, [], )
    assert e.value.status == mw.MW_ERR_INVALID_ARG
    with pytest.raises(mw.MWError) as e:
        mw.mw_engine_create(0, [64] * 17)
    assert e.value.status == mw.MW_ERR_INVALID_ARG
    with pytest.raises(mw.MWError) as e:
        mw.mw_engine_streams(None, 0)
    assert e.value.status == mw.MW_ERR_INVALID_ARG
    with pytest.raises(mw.MWError) as e:
        mw.mw_engine_memory(None)
    assert e.value.status == mw.MW_ERR_INVALID_ARG
    mw.mw_engine_destroy(None)
    plan = mw.EnginePlan(0, 1, 1, 1, 1, mw.MW_ENGINE_POLLED, 1)
    dec = dict(pool=None, hq=8, hkv=2, head_dim=128, scale=0.1, seq_lens=[5], d_seq_lens=0, d_block_table=0,
               bt_stride=1, d_q=0, d_out=0, d_workspace=0, workspace_bytes=0)
    pre = dict(pool=None, hq=8, hkv=2, head_dim=128, scale=0.1, new_lens=[5], prefix_lens=[0], d_qo_indptr=0,
               d_prefix_lens=0, d_block_table=0, bt_stride=1, d_q=0, d_out=0)
    with pytest.raises(mw.MWError) as e:
        mw.mw_engine_run(None, dec, pre, plan)
    assert e.value.status == mw.MW_ERR_INVALID_ARG


def test_engine_structs_match_the_header(tmp_path):
    """ctypes layouts of the engine's argument, plan and stats structs agree
    with what a C compiler makes of the header."""
    import subprocess
    structs = {"mw_decode_args": mw._DecodeArgs, "mw_prefill_args": mw._PrefillArgs,
               "mw_engine_plan": mw.EnginePlan, "mw_engine_stats": mw.EngineStats}
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "mw.h"', "int main(void) {"]
    for cname, cls in structs.items():
        lines.append(f'printf("{cname} size %zu\\n", sizeof({cname}));')
        for f, _ in cls._fields_:
            lines.append(f'printf("{cname} {f} %zu\\n", offsetof({cname}, {f}));')
    lines.append("return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    inc = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
    subprocess.run(["gcc", "-std=c11", "-I", inc, str(src), "-o", str(exe)], check=True)
    got = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    for line in filter(None, got):
        cname, field, val = line.split()
        cls = structs[cname]
        want = ctypes.sizeof(cls) if field == "size" else getattr(cls, field).offset
        assert int(val) == want, (cname, field, val, want)


def test_decode_workspace_covers_both_splits():
    """The workspace size for chunk_pages 0 fits the balanced split on any
    stream and the fixed chunks that the fused call takes for 0."""
    from paper_2504_14489_amd import mw, workloads as W
    lens = W.make_workload(W.custom_config(hq=32, hkv=8, pre_chunks=((0, 1),), dec_batch=64,
                                           dec_len_lo=1, dec_len_hi=4096, seed=3)).dec_lens
    size0 = mw.mw_decode_workspace_size(32, 8, 128, lens, 0)
    assert size0 >= mw.mw_decode_workspace_size(32, 8, 128, lens, -1)
    # largest balanced split: 512 ranges, a piece of each (range, segment)
    # boundary: (512 + 64 * 8 - 1) slots of 4 heads x 128 fp32 + (m, l)
    assert size0 >= (512 + 64 * 8 - 1) * 4 * (128 * 4 + 8)
