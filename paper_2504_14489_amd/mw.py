"""Python binding of the C ABI in include/mw.h (argument marshalling only).

Every function here has the name of the C entry point it calls and does no
arithmetic of its own: device buffers are passed as integer addresses (for
torch tensors, ``t.data_ptr()``), host arrays as numpy int32 arrays, streams
as integer hipStream_t handles (``torch.cuda.current_stream().cuda_stream``).
A failing call raises :class:`MWError` carrying the status and the library's
error text.

The library must have been built (``python -m paper_2504_14489_amd.build``);
there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmw.so")

MW_OK = 0
MW_ERR_INVALID_ARG = -1
MW_ERR_UNSUPPORTED = -2
MW_ERR_OUT_OF_PAGES = -3
MW_ERR_HIP = -4
MW_ERR_NOT_READY = -5


class MWError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"[{status}] {message}")
        self.status = status
        self.message = message


class _PoolDesc(ctypes.Structure):
    _fields_ = [("num_pages", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32)]


class GuardKey(ctypes.Structure):
    """mw_guard_key: the five variables of a contention-guard cell."""
    _fields_ = [("prefill_new", ctypes.c_int64), ("prefill_reused", ctypes.c_int64),
                ("decode_batch", ctypes.c_int64), ("decode_reused", ctypes.c_int64),
                ("prefill_cus", ctypes.c_int32)]


class _AttnShape(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("scale", ctypes.c_float)]


class _DecodeArgs(ctypes.Structure):
    _fields_ = [("pool", ctypes.c_void_p), ("shape", _AttnShape), ("batch", ctypes.c_int32),
                ("h_seq_lens", ctypes.c_void_p), ("d_seq_lens", ctypes.c_void_p),
                ("d_block_table", ctypes.c_void_p), ("bt_stride", ctypes.c_int32),
                ("d_q", ctypes.c_void_p), ("d_out", ctypes.c_void_p), ("d_workspace", ctypes.c_void_p),
                ("workspace_bytes", ctypes.c_size_t), ("chunk_pages", ctypes.c_int32)]


class _PrefillArgs(ctypes.Structure):
    _fields_ = [("pool", ctypes.c_void_p), ("shape", _AttnShape), ("batch", ctypes.c_int32),
                ("h_new_lens", ctypes.c_void_p), ("h_prefix_lens", ctypes.c_void_p),
                ("d_qo_indptr", ctypes.c_void_p), ("d_prefix_lens", ctypes.c_void_p),
                ("d_block_table", ctypes.c_void_p), ("bt_stride", ctypes.c_int32),
                ("d_q", ctypes.c_void_p), ("d_out", ctypes.c_void_p),
                ("d_workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t)]


class EnginePlan(ctypes.Structure):
    """mw_engine_plan (policy: MW_ENGINE_BLOCKING or MW_ENGINE_POLLED)."""
    _fields_ = [("config", ctypes.c_int32), ("decode_iters", ctypes.c_int32),
                ("decode_layers", ctypes.c_int32), ("prefill_layers", ctypes.c_int32),
                ("layers_per_launch", ctypes.c_int32), ("policy", ctypes.c_int32),
                ("switch_on_decode_end", ctypes.c_int32), ("decode_graph", ctypes.c_int32)]


class EngineStats(ctypes.Structure):
    _fields_ = [(f, ctypes.c_double) for f in (
        "wall_ms", "decode_busy_ms", "prefill_busy_ms", "decode_bubble", "prefill_bubble", "bubble_ratio",
        "decode_gap_ms_max", "decode_iter_ms_mean", "prefill_end_ms", "switch_gap_ms", "switch_host_us",
        "host_launch_ms", "decode_launch_us_mean")] + [("prefill_batches", ctypes.c_int32), ("switched_layers", ctypes.c_int32)]

    def as_dict(self) -> dict:
        return {f: getattr(self, f) for f, _ in self._fields_}


MW_ENGINE_BLOCKING = 0
MW_ENGINE_POLLED = 1

_lib = None
_P = ctypes.c_void_p
_I = ctypes.c_int32
_PI = ctypes.POINTER(ctypes.c_int32)
_PU = ctypes.POINTER(ctypes.c_uint32)
_PF = ctypes.POINTER(ctypes.c_float)
_PD = ctypes.POINTER(ctypes.c_double)

_SIGNATURES = {
    "mw_last_error": ([], ctypes.c_char_p),
    "mw_version": ([], _I),
    "mw_sync": ([_P], _I),
    "mw_kv_pool_create": ([ctypes.POINTER(_PoolDesc), _P, _P, ctypes.POINTER(_P)], _I),
    "mw_kv_pool_destroy": ([_P], _I),
    "mw_kv_pool_set_free_order": ([_P, _PI, _I], _I),
    "mw_kv_pool_alloc": ([_P, _I, _PI], _I),
    "mw_kv_pool_free": ([_P, _PI, _I], _I),
    "mw_kv_pool_num_free": ([_P, _PI], _I),
    "mw_kv_pool_write": ([_P, _I, _PI, _PI, _P, _P, _P, _I, _P, _P, _P, _P], _I),
    "mw_kv_pool_gather": ([_P, _P, _I, _P, _P, _P], _I),
    "mw_partition_create": ([_I, _I, _I, ctypes.POINTER(_P)], _I),
    "mw_partition_create_masks": ([_I, _PU, _PU, _I, ctypes.POINTER(_P)], _I),
    "mw_partition_streams": ([_P, ctypes.POINTER(_P), ctypes.POINTER(_P)], _I),
    "mw_partition_masks": ([_P, _PU, _PU], _I),
    "mw_partition_destroy": ([_P], _I),
    "mw_cu_probe": ([_I, _I, _P, _P, _P], _I),
    "mw_cache_flush": ([_P, ctypes.c_size_t, _P], _I),
    "mw_mfma_peak": ([_I, _I, _P, _P, _P, ctypes.POINTER(ctypes.c_double)], _I),
    "mw_trace_mark": ([_I, _P], _I),
    "mw_stream_read": ([_P, ctypes.c_size_t, _P, _I, _P, _P], _I),
    "mw_timing_create": ([ctypes.POINTER(_P)], _I),
    "mw_timing_destroy": ([_P], _I),
    "mw_timing_mark": ([_P, _P], _I),
    "mw_timing_elapsed": ([_P, _PF, _PF], _I),
    "mw_timing_kernels": ([_P, _PI], _I),
    "mw_timing_kernel_ms": ([_P, _I, _PF], _I),
    "mw_timing_offsets": ([_P, _P, _PF, _PF], _I),
    "mw_prefill_attn": ([_P, ctypes.POINTER(_AttnShape), _I, _PI, _PI, _P, _P, _P, _I, _P, _P, _P,
                         _P], _I),
    "mw_prefill_workspace_size": ([ctypes.POINTER(_AttnShape), _I, _PI, _PI, _I,
                                   ctypes.POINTER(ctypes.c_size_t)], _I),
    "mw_prefill_attn_ws": ([_P, ctypes.POINTER(_AttnShape), _I, _PI, _PI, _P, _P, _P, _I, _P, _P, _P,
                            ctypes.c_size_t, _P, _P], _I),
    "mw_decode_workspace_size": ([ctypes.POINTER(_AttnShape), _I, _PI, _I,
                                  ctypes.POINTER(ctypes.c_size_t)], _I),
    "mw_decode_attn": ([_P, ctypes.POINTER(_AttnShape), _I, _PI, _P, _P, _I, _P, _P, _P,
                        ctypes.c_size_t, _I, _P, _P], _I),
    "mw_decode_attn_noalloc": ([_P, ctypes.POINTER(_AttnShape), _I, _PI, _P, _P, _I, _P, _P, _I, _P], _I),
    "mw_predictor_create": ([ctypes.POINTER(_P)], _I),
    "mw_predictor_destroy": ([_P], _I),
    "mw_predictor_set_launch_shape": ([_P, _I, _I], _I),
    "mw_predictor_add_prefill": ([_P, _I, _I, _PI, _PI, ctypes.c_double], _I),
    "mw_predictor_add_decode": ([_P, _I, _I, _PI, ctypes.c_double], _I),
    "mw_predictor_fit": ([_P], _I),
    "mw_predictor_prefill_ms": ([_P, _I, _I, _PI, _PI, _PD], _I),
    "mw_predictor_decode_ms": ([_P, _I, _I, _PI, _PD], _I),
    "mw_predictor_coefficients": ([_P, _I, _I, _PD], _I),
    "mw_guard_create": ([ctypes.POINTER(_P)], _I),
    "mw_guard_destroy": ([_P], _I),
    "mw_guard_add": ([_P, ctypes.POINTER(GuardKey), ctypes.c_double], _I),
    "mw_guard_lookup": ([_P, ctypes.POINTER(GuardKey), _PD], _I),
    "mw_prefill_layers": ([ctypes.c_double, ctypes.c_double, _I, _PI], _I),
    "mw_engine_create": ([_I, _PI, _I, ctypes.POINTER(_P)], _I),
    "mw_engine_destroy": ([_P], _I),
    "mw_engine_streams": ([_P, _I, ctypes.POINTER(_P), ctypes.POINTER(_P)], _I),
    "mw_engine_memory": ([_P, ctypes.POINTER(ctypes.c_int64), _PD], _I),
    "mw_engine_run": ([_P, ctypes.POINTER(_DecodeArgs), ctypes.POINTER(_PrefillArgs),
                       ctypes.POINTER(EnginePlan), ctypes.POINTER(EngineStats)], _I),
    "mw_engine_timeline": ([_P, _I, _PD, _I, _PI], _I),
    "mw_engine_graphs": ([_P, _PI, ctypes.POINTER(ctypes.c_int64), _PD], _I),
    "mw_fused_attn": ([ctypes.POINTER(_PrefillArgs), ctypes.POINTER(_DecodeArgs), _P, _P], _I),
}

EXPORTED = tuple(_SIGNATURES)


def load(path: str = LIB_PATH):
    """Loads libmw.so (raising if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with `python -m paper_2504_14489_amd.build`")
        lib = ctypes.CDLL(path)
        for name, (args, res) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.argtypes = args
            fn.restype = res
        _lib = lib
    return _lib


def _check(st: int):
    if st != MW_OK:
        raise MWError(st, mw_last_error())


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32).reshape(-1))


def _pi(a: np.ndarray):
    return a.ctypes.data_as(_PI)


def _shape(hq: int, hkv: int, head_dim: int, scale: float) -> _AttnShape:
    return _AttnShape(int(hq), int(hkv), int(head_dim), float(scale))


def _h(x) -> Optional[int]:
    """A handle or device address as an int (None stays NULL)."""
    if x is None:
        return None
    if isinstance(x, ctypes.c_void_p):
        return x.value
    return int(x)


# ------------------------------------------------------------------ misc ---
def mw_last_error() -> str:
    return load().mw_last_error().decode()


def mw_version() -> int:
    return load().mw_version()


def mw_sync(stream=0):
    _check(load().mw_sync(_h(stream)))


# ------------------------------------------------------------------ pool ---
def mw_kv_pool_create(num_pages: int, page_size: int, num_kv_heads: int, head_dim: int,
                      d_k_pages: int, d_v_pages: int):
    out = _P()
    desc = _PoolDesc(num_pages, page_size, num_kv_heads, head_dim)
    _check(load().mw_kv_pool_create(ctypes.byref(desc), _h(d_k_pages), _h(d_v_pages),
                                    ctypes.byref(out)))
    return out


def mw_kv_pool_destroy(pool):
    _check(load().mw_kv_pool_destroy(pool))


def mw_kv_pool_set_free_order(pool, perm):
    p = _i32(perm)
    _check(load().mw_kv_pool_set_free_order(pool, _pi(p), len(p)))


def mw_kv_pool_alloc(pool, n_pages: int) -> np.ndarray:
    out = np.zeros(max(n_pages, 1), dtype=np.int32)
    _check(load().mw_kv_pool_alloc(pool, n_pages, _pi(out)))
    return out[:n_pages]


def mw_kv_pool_free(pool, pages):
    p = _i32(pages)
    _check(load().mw_kv_pool_free(pool, _pi(p), len(p)))


def mw_kv_pool_num_free(pool) -> int:
    n = ctypes.c_int32()
    _check(load().mw_kv_pool_num_free(pool, ctypes.byref(n)))
    return n.value


def mw_kv_pool_write(pool, new_lens, start_pos, d_qo_indptr: int, d_start_pos: int,
                     d_block_table: int, bt_stride: int, d_k_new: int, d_v_new: int,
                     stream=0, timing=None):
    nl, sp = _i32(new_lens), _i32(start_pos)
    _check(load().mw_kv_pool_write(pool, len(nl), _pi(nl), _pi(sp), _h(d_qo_indptr),
                                   _h(d_start_pos), _h(d_block_table), bt_stride, _h(d_k_new),
                                   _h(d_v_new), _h(stream), timing))


def mw_kv_pool_gather(pool, d_block_table: int, n_tokens: int, d_k_out: int, d_v_out: int,
                      stream=0):
    _check(load().mw_kv_pool_gather(pool, _h(d_block_table), n_tokens, _h(d_k_out),
                                    _h(d_v_out), _h(stream)))


# ------------------------------------------------------------- partition ---
def mw_partition_create(device: int, prefill_cus: int, decode_cus: int):
    out = _P()
    _check(load().mw_partition_create(device, prefill_cus, decode_cus, ctypes.byref(out)))
    return out


def mw_partition_create_masks(device: int, prefill_mask, decode_mask):
    pm = np.ascontiguousarray(prefill_mask, dtype=np.uint32)
    dm = np.ascontiguousarray(decode_mask, dtype=np.uint32)
    assert len(pm) == len(dm)
    out = _P()
    _check(load().mw_partition_create_masks(device, pm.ctypes.data_as(_PU), dm.ctypes.data_as(_PU),
                                            len(pm), ctypes.byref(out)))
    return out


def mw_partition_streams(part) -> Tuple[int, int]:
    p, d = _P(), _P()
    _check(load().mw_partition_streams(part, ctypes.byref(p), ctypes.byref(d)))
    return p.value or 0, d.value or 0


def mw_partition_masks(part) -> Tuple[np.ndarray, np.ndarray]:
    pm = np.zeros(8, dtype=np.uint32)
    dm = np.zeros(8, dtype=np.uint32)
    _check(load().mw_partition_masks(part, pm.ctypes.data_as(_PU), dm.ctypes.data_as(_PU)))
    return pm, dm


def mw_partition_destroy(part):
    _check(load().mw_partition_destroy(part))


def mw_cu_probe(n_blocks: int, spin_cycles: int, d_out: int, stream=0, timing=None):
    _check(load().mw_cu_probe(n_blocks, spin_cycles, _h(d_out), _h(stream), timing))


def mw_cache_flush(d_buf: int, nbytes: int, stream=0):
    _check(load().mw_cache_flush(_h(d_buf), nbytes, _h(stream)))


def mw_mfma_peak(n_blocks: int, iters: int, d_sink: int, stream=0, timing=None) -> float:
    """Launches the matrix-core probe; returns its floating-point operations."""
    flop = ctypes.c_double()
    _check(load().mw_mfma_peak(n_blocks, iters, _h(d_sink), _h(stream), timing, ctypes.byref(flop)))
    return flop.value


def mw_trace_mark(mark_id: int, stream=0):
    _check(load().mw_trace_mark(mark_id, _h(stream)))


def mw_stream_read(d_src: int, nbytes: int, d_sink: int, n_blocks: int, stream=0, timing=None):
    _check(load().mw_stream_read(_h(d_src), nbytes, _h(d_sink), n_blocks, _h(stream), timing))


# ---------------------------------------------------------------- timing ---
def mw_timing_create():
    out = _P()
    _check(load().mw_timing_create(ctypes.byref(out)))
    return out


def mw_timing_destroy(t):
    _check(load().mw_timing_destroy(t))


def mw_timing_mark(t, stream=0):
    _check(load().mw_timing_mark(t, _h(stream)))


def mw_timing_elapsed(t) -> Tuple[float, float]:
    g, h = ctypes.c_float(), ctypes.c_float()
    _check(load().mw_timing_elapsed(t, ctypes.byref(g), ctypes.byref(h)))
    return g.value, h.value


def mw_timing_kernels(t) -> int:
    n = ctypes.c_int32()
    _check(load().mw_timing_kernels(t, ctypes.byref(n)))
    return n.value


def mw_timing_kernel_ms(t, k: int) -> float:
    ms = ctypes.c_float()
    _check(load().mw_timing_kernel_ms(t, k, ctypes.byref(ms)))
    return ms.value


def mw_timing_offsets(t, ref) -> Tuple[float, float]:
    a, b = ctypes.c_float(), ctypes.c_float()
    _check(load().mw_timing_offsets(t, ref, ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


# ------------------------------------------------------------- attention ---
def mw_prefill_attn(pool, num_q_heads: int, num_kv_heads: int, head_dim: int, scale: float,
                    new_lens, prefix_lens, d_qo_indptr: int, d_prefix_lens: int,
                    d_block_table: int, bt_stride: int, d_q: int, d_out: int, stream=0,
                    timing=None):
    nl, pl = _i32(new_lens), _i32(prefix_lens)
    sh = _shape(num_q_heads, num_kv_heads, head_dim, scale)
    _check(load().mw_prefill_attn(pool, ctypes.byref(sh), len(nl), _pi(nl), _pi(pl),
                                  _h(d_qo_indptr), _h(d_prefix_lens), _h(d_block_table), bt_stride,
                                  _h(d_q), _h(d_out), _h(stream), timing))


def mw_prefill_workspace_size(num_q_heads: int, num_kv_heads: int, head_dim: int, new_lens,
                              prefix_lens, num_cus: int = 0) -> int:
    nl, pl = _i32(new_lens), _i32(prefix_lens)
    sh = _shape(num_q_heads, num_kv_heads, head_dim, 1.0)
    out = ctypes.c_size_t()
    _check(load().mw_prefill_workspace_size(ctypes.byref(sh), len(nl), _pi(nl), _pi(pl), num_cus,
                                            ctypes.byref(out)))
    return out.value


def mw_prefill_attn_ws(pool, num_q_heads: int, num_kv_heads: int, head_dim: int, scale: float,
                       new_lens, prefix_lens, d_qo_indptr: int, d_prefix_lens: int,
                       d_block_table: int, bt_stride: int, d_q: int, d_out: int, d_workspace: int,
                       workspace_bytes: int, stream=0, timing=None):
    nl, pl = _i32(new_lens), _i32(prefix_lens)
    sh = _shape(num_q_heads, num_kv_heads, head_dim, scale)
    _check(load().mw_prefill_attn_ws(pool, ctypes.byref(sh), len(nl), _pi(nl), _pi(pl),
                                     _h(d_qo_indptr), _h(d_prefix_lens), _h(d_block_table), bt_stride,
                                     _h(d_q), _h(d_out), _h(d_workspace), workspace_bytes, _h(stream),
                                     timing))


def mw_decode_workspace_size(num_q_heads: int, num_kv_heads: int, head_dim: int, seq_lens,
                             chunk_pages: int = 0) -> int:
    sl = _i32(seq_lens)
    sh = _shape(num_q_heads, num_kv_heads, head_dim, 1.0)
    out = ctypes.c_size_t()
    _check(load().mw_decode_workspace_size(ctypes.byref(sh), len(sl), _pi(sl), chunk_pages,
                                           ctypes.byref(out)))
    return out.value


def mw_decode_attn(pool, num_q_heads: int, num_kv_heads: int, head_dim: int, scale: float,
                   seq_lens, d_seq_lens: int, d_block_table: int, bt_stride: int, d_q: int,
                   d_out: int, d_workspace: int, workspace_bytes: int, chunk_pages: int = 0,
                   stream=0, timing=None):
    sl = _i32(seq_lens)
    sh = _shape(num_q_heads, num_kv_heads, head_dim, scale)
    _check(load().mw_decode_attn(pool, ctypes.byref(sh), len(sl), _pi(sl), _h(d_seq_lens),
                                 _h(d_block_table), bt_stride, _h(d_q), _h(d_out), _h(d_workspace),
                                 workspace_bytes, chunk_pages, _h(stream), timing))


def mw_decode_attn_noalloc(pool, num_q_heads: int, num_kv_heads: int, head_dim: int, scale: float,
                           seq_lens, d_seq_lens: int, d_block_table: int, bt_stride: int, d_q: int,
                           d_out: int, chunk_pages: int = 0, stream=0):
    sl = _i32(seq_lens)
    sh = _shape(num_q_heads, num_kv_heads, head_dim, scale)
    _check(load().mw_decode_attn_noalloc(pool, ctypes.byref(sh), len(sl), _pi(sl), _h(d_seq_lens),
                                         _h(d_block_table), bt_stride, _h(d_q), _h(d_out), chunk_pages,
                                         _h(stream)))


# ---- contention-tolerant estimator (host-side)

def mw_predictor_create():
    p = _P()
    _check(load().mw_predictor_create(ctypes.byref(p)))
    return p


def mw_predictor_destroy(p):
    _check(load().mw_predictor_destroy(p))


def mw_predictor_set_launch_shape(p, num_q_heads: int, num_kv_heads: int):
    _check(load().mw_predictor_set_launch_shape(p, int(num_q_heads), int(num_kv_heads)))


def mw_predictor_add_prefill(p, cus: int, new_lens, prefix_lens, ms: float):
    n, r = _i32(new_lens), _i32(prefix_lens)
    if len(n) != len(r):
        raise ValueError("new_lens and prefix_lens differ in length")
    _check(load().mw_predictor_add_prefill(p, cus, len(n), _pi(n), _pi(r), ms))


def mw_predictor_add_decode(p, cus: int, seq_lens, ms: float):
    lens = _i32(seq_lens)
    _check(load().mw_predictor_add_decode(p, cus, len(lens), _pi(lens), ms))


def mw_predictor_fit(p):
    _check(load().mw_predictor_fit(p))


def mw_predictor_prefill_ms(p, cus: int, new_lens, prefix_lens) -> float:
    n, r = _i32(new_lens), _i32(prefix_lens)
    if len(n) != len(r):
        raise ValueError("new_lens and prefix_lens differ in length")
    out = ctypes.c_double()
    _check(load().mw_predictor_prefill_ms(p, cus, len(n), _pi(n), _pi(r), ctypes.byref(out)))
    return out.value


def mw_predictor_decode_ms(p, cus: int, seq_lens) -> float:
    lens = _i32(seq_lens)
    out = ctypes.c_double()
    _check(load().mw_predictor_decode_ms(p, cus, len(lens), _pi(lens), ctypes.byref(out)))
    return out.value


def mw_predictor_coefficients(p, phase: int, cus: int) -> np.ndarray:
    th = (ctypes.c_double * 4)()
    _check(load().mw_predictor_coefficients(p, phase, cus, th))
    return np.array(th[:], dtype=np.float64)


def mw_guard_create():
    g = _P()
    _check(load().mw_guard_create(ctypes.byref(g)))
    return g


def mw_guard_destroy(g):
    _check(load().mw_guard_destroy(g))


def mw_guard_add(g, prefill_new: int, prefill_reused: int, decode_batch: int, decode_reused: int,
                 prefill_cus: int, slowdown: float):
    key = GuardKey(prefill_new, prefill_reused, decode_batch, decode_reused, prefill_cus)
    _check(load().mw_guard_add(g, ctypes.byref(key), slowdown))


def mw_guard_lookup(g, prefill_new: int, prefill_reused: int, decode_batch: int, decode_reused: int,
                    prefill_cus: int) -> float:
    key = GuardKey(prefill_new, prefill_reused, decode_batch, decode_reused, prefill_cus)
    out = ctypes.c_double()
    _check(load().mw_guard_lookup(g, ctypes.byref(key), ctypes.byref(out)))
    return out.value


def mw_prefill_layers(t_decode_ms: float, t_prefill_ms: float, n_layers: int) -> int:
    out = ctypes.c_int32()
    _check(load().mw_prefill_layers(t_decode_ms, t_prefill_ms, n_layers, ctypes.byref(out)))
    return out.value


# ---- multiplex engine

def mw_engine_create(device: int, prefill_cus) -> ctypes.c_void_p:
    pc = _i32(prefill_cus)
    out = _P()
    _check(load().mw_engine_create(device, _pi(pc), len(pc), ctypes.byref(out)))
    return out


def mw_engine_destroy(eng):
    _check(load().mw_engine_destroy(eng))


def mw_engine_streams(eng, config: int) -> Tuple[int, int]:
    p, d = _P(), _P()
    _check(load().mw_engine_streams(eng, config, ctypes.byref(p), ctypes.byref(d)))
    return p.value or 0, d.value or 0


def mw_engine_memory(eng) -> Tuple[int, float]:
    b, ms = ctypes.c_int64(), ctypes.c_double()
    _check(load().mw_engine_memory(eng, ctypes.byref(b), ctypes.byref(ms)))
    return b.value, ms.value


def _engine_structs(dec: dict, pre: dict):
    """ctypes argument structs (and the host arrays they point at) from dicts."""
    sl = _i32(dec["seq_lens"])
    nl, pl = _i32(pre["new_lens"]), _i32(pre["prefix_lens"])
    da = _DecodeArgs(_h(dec["pool"]), _shape(dec["hq"], dec["hkv"], dec["head_dim"], dec["scale"]), len(sl),
                     sl.ctypes.data, _h(dec["d_seq_lens"]), _h(dec["d_block_table"]), dec["bt_stride"],
                     _h(dec["d_q"]), _h(dec["d_out"]), _h(dec["d_workspace"]), dec["workspace_bytes"],
                     dec.get("chunk_pages", 0))
    pa = _PrefillArgs(_h(pre["pool"]), _shape(pre["hq"], pre["hkv"], pre["head_dim"], pre["scale"]), len(nl),
                      nl.ctypes.data, pl.ctypes.data, _h(pre["d_qo_indptr"]), _h(pre["d_prefix_lens"]),
                      _h(pre["d_block_table"]), pre["bt_stride"], _h(pre["d_q"]), _h(pre["d_out"]),
                      _h(pre.get("d_workspace")), pre.get("workspace_bytes", 0))
    return da, pa, (sl, nl, pl)


def mw_fused_attn(pre: dict, dec: dict, stream=0, timing=None):
    """One fused prefill + decode launch; dicts as for :func:`mw_engine_run`."""
    da, pa, keep = _engine_structs(dec, pre)
    _check(load().mw_fused_attn(ctypes.byref(pa), ctypes.byref(da), _h(stream), _h(timing)))


def mw_engine_run(eng, dec: dict, pre: dict, plan: EnginePlan) -> dict:
    """dec: pool, hq, hkv, head_dim, scale, seq_lens (host), d_seq_lens, d_block_table,
    bt_stride, d_q, d_out, d_workspace, workspace_bytes, chunk_pages;
    pre: pool, hq, hkv, head_dim, scale, new_lens, prefix_lens (host), d_qo_indptr,
    d_prefix_lens, d_block_table, bt_stride, d_q, d_out.  Returns the stats as a dict."""
    da, pa, keep = _engine_structs(dec, pre)
    st = EngineStats()
    _check(load().mw_engine_run(eng, ctypes.byref(da), ctypes.byref(pa), ctypes.byref(plan), ctypes.byref(st)))
    return st.as_dict()


def mw_engine_timeline(eng, phase: int) -> np.ndarray:
    """[n_calls][3] float64: start ms, end ms, on-whole-device flag."""
    n = ctypes.c_int32()
    _check(load().mw_engine_timeline(eng, phase, None, 0, ctypes.byref(n)))
    out = np.zeros((n.value, 3), dtype=np.float64)
    if n.value:
        _check(load().mw_engine_timeline(eng, phase, out.ctypes.data_as(_PD), n.value, ctypes.byref(n)))
    return out


def mw_engine_graphs(eng) -> Tuple[int, int, float]:
    """(number of captured decode graphs, their device bytes, capture ms)."""
    n, b, ms = ctypes.c_int32(), ctypes.c_int64(), ctypes.c_double()
    _check(load().mw_engine_graphs(eng, ctypes.byref(n), ctypes.byref(b), ctypes.byref(ms)))
    return n.value, b.value, ms.value
