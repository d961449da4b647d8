"""CPU oracle for paged grouped-query attention (test infrastructure).

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg use this package.  The library's GPU path neither imports nor links it.

The arithmetic lives in ``mw_oracle.c`` (plain C, double precision); this file
only compiles it with gcc and marshals numpy arrays.  Row semantics:

* prefill token i of a chunk with cached prefix r sees keys 0 .. r+i
  (``nvis = r + i + 1``): the paper's prefill with cache attends L = r + n keys
  (Sec. 3.3, Table "tab:theory_cost") and a chunk reads the KV of all earlier
  chunks (Sec. 1);
* a decode token of a sequence with L cached tokens (its own K/V already
  written at position L-1) sees keys 0 .. L-1, the r + 1 keys of the same
  table.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
import subprocess
from typing import Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mw_oracle.c")
_LIB = os.path.join(_HERE, "libmw_oracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no HIP, no vendor math libraries)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fPIC",
                               "-shared", "-pthread", "-Wall", "-Wextra", "-o", tmp, _SRC,
                               "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load(path: Optional[str] = None):
    global _lib
    if _lib is None:
        if path is None:
            build(force=False)
        lib = ctypes.CDLL(path or _LIB)
        P = ctypes.c_void_p
        i32 = ctypes.c_int32
        lib.mwo_paged_attention.argtypes = [i32, i32, i32, i32, i32, ctypes.c_double, P, P, P,
                                            i32, P, i32, P, P, P, P, i32, i32]
        lib.mwo_paged_attention.restype = i32
        lib.mwo_merge_parts.argtypes = [i32, i32, P, P, P, P]
        lib.mwo_merge_parts.restype = i32
        lib.mwo_partial.argtypes = [i32, i32, i32, i32, ctypes.c_double, P, P, P, i32, P, i32,
                                    i32, i32, P, P, P]
        lib.mwo_partial.restype = i32
        _lib = lib
    return _lib


@contextlib.contextmanager
def use_library(path: str):
    """Temporarily route every oracle call through another build of the
    oracle (used by the test that plants mistakes in a copy of its source)."""
    global _lib
    saved = _lib
    _lib = None
    _load(path)
    try:
        yield
    finally:
        _lib = saved


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def default_threads() -> int:
    """Host threads the oracle uses by default: the CPUs this process may run
    on, capped by OMP_NUM_THREADS when that is set (a machine's share of its
    cores for one job) and by 64."""
    try:
        n = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        n = os.cpu_count() or 1
    try:
        n = min(n, int(os.environ.get("OMP_NUM_THREADS", n)))
    except ValueError:
        pass
    return max(1, min(n, 64))


def paged_attention(q: np.ndarray, k_pool: np.ndarray, v_pool: np.ndarray,
                    block_tables: np.ndarray, row_table: Sequence[int],
                    row_nvis: Sequence[int], hkv: Optional[int] = None,
                    scale: Optional[float] = None, n_threads: Optional[int] = None,
                    want_probs: bool = False):
    """Attention for independent rows.

    q: uint16 [rows][Hq][D]; pools: uint16 [P][Hkv][S][D];
    block_tables: int32 [T][stride] (or 1-D for a single table);
    row_table[r]: which table row r uses; row_nvis[r]: visible keys.
    Returns float64 [rows][Hq][D] (and [rows][Hq][max nvis] softmax weights
    when ``want_probs``).
    """
    lib = _load()
    q = np.ascontiguousarray(q, dtype=np.uint16)
    k_pool = np.ascontiguousarray(k_pool, dtype=np.uint16)
    v_pool = np.ascontiguousarray(v_pool, dtype=np.uint16)
    bt = np.ascontiguousarray(np.atleast_2d(block_tables), dtype=np.int32)
    row_table = np.ascontiguousarray(row_table, dtype=np.int32)
    row_nvis = np.ascontiguousarray(row_nvis, dtype=np.int32)
    n_rows, hq, d = q.shape
    P, hkv_pool, s, d2 = k_pool.shape
    if hkv is None:
        hkv = hkv_pool
    assert d == d2 and hkv == hkv_pool and v_pool.shape == k_pool.shape
    assert len(row_table) == n_rows and len(row_nvis) == n_rows
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    out = np.zeros((n_rows, hq, d), dtype=np.float64)
    probs = None
    pstride = 0
    if want_probs:
        pstride = int(max(row_nvis.max(initial=1), 1))
        probs = np.zeros((n_rows, hq, pstride), dtype=np.float64)
    st = lib.mwo_paged_attention(n_rows, hq, hkv, d, s, float(scale), _ptr(q), _ptr(k_pool),
                                 _ptr(v_pool), P, _ptr(bt), bt.shape[1], _ptr(row_table),
                                 _ptr(row_nvis), _ptr(out),
                                 _ptr(probs) if probs is not None else None, pstride,
                                 n_threads or default_threads())
    if st != 0:
        raise ValueError(f"oracle rejected its arguments (status {st})")
    return (out, probs) if want_probs else out


def prefill(q_rows: np.ndarray, k_pool, v_pool, bt: np.ndarray, prefix_len: int,
            scale: Optional[float] = None, n_threads: Optional[int] = None,
            want_probs: bool = False):
    """Causal prefill of n = len(q_rows) new tokens over a cached prefix of
    ``prefix_len`` tokens; row i sees keys 0 .. prefix_len + i."""
    n = q_rows.shape[0]
    nvis = prefix_len + 1 + np.arange(n, dtype=np.int32)
    return paged_attention(q_rows, k_pool, v_pool, np.asarray(bt)[None, :],
                           np.zeros(n, dtype=np.int32), nvis, scale=scale,
                           n_threads=n_threads, want_probs=want_probs)


def decode(q: np.ndarray, k_pool, v_pool, bt: np.ndarray, seq_lens,
           scale: Optional[float] = None, n_threads: Optional[int] = None,
           want_probs: bool = False):
    """Decode: sequence b's query sees its L_b cached keys 0 .. L_b - 1."""
    B = q.shape[0]
    return paged_attention(q, k_pool, v_pool, bt, np.arange(B, dtype=np.int32),
                           np.asarray(seq_lens, dtype=np.int32), scale=scale,
                           n_threads=n_threads, want_probs=want_probs)


def partial(q_row: np.ndarray, k_pool, v_pool, bt: np.ndarray, head: int, j0: int, j1: int,
            scale: Optional[float] = None) -> Tuple[float, float, np.ndarray]:
    """(m, l, unnormalised o) of one head over keys [j0, j1)."""
    lib = _load()
    q_row = np.ascontiguousarray(q_row, dtype=np.uint16)
    k_pool = np.ascontiguousarray(k_pool, dtype=np.uint16)
    v_pool = np.ascontiguousarray(v_pool, dtype=np.uint16)
    bt = np.ascontiguousarray(bt, dtype=np.int32)
    hq, d = q_row.shape
    P, hkv, s, _ = k_pool.shape
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    m = np.zeros(1)
    l = np.zeros(1)
    o = np.zeros(d)
    st = lib.mwo_partial(hq, hkv, d, s, float(scale), _ptr(q_row), _ptr(k_pool), _ptr(v_pool),
                         P, _ptr(bt), head, j0, j1, _ptr(m), _ptr(l), _ptr(o))
    if st != 0:
        raise ValueError(f"oracle rejected its arguments (status {st})")
    return float(m[0]), float(l[0]), o


def merge_parts(m: Sequence[float], l: Sequence[float], o: np.ndarray) -> np.ndarray:
    """Log-sum-exp merge of partial results over disjoint key sets."""
    lib = _load()
    m = np.ascontiguousarray(m, dtype=np.float64)
    l = np.ascontiguousarray(l, dtype=np.float64)
    o = np.ascontiguousarray(o, dtype=np.float64)
    out = np.zeros(o.shape[1])
    st = lib.mwo_merge_parts(len(m), o.shape[1], _ptr(m), _ptr(l), _ptr(o), _ptr(out))
    if st != 0:
        raise ValueError("every part is empty")
    return out
