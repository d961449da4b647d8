"""A synthetic workload resident in GPU memory, driven through the C ABI.

Glue used by the tests, the benchmark and the smoke check: torch allocates
the device buffers (pools, block tables, Q, O, workspaces) and every step of
the attention path runs in the library's HIP kernels via :mod:`.mw`.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence, Tuple

import numpy as np
import torch

from . import mw
from .workloads import Workload


def _dev16(a: np.ndarray, device) -> torch.Tensor:
    """uint16 numpy -> int16 device tensor with the same bits."""
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device)


def _dev32(a, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.int32))).to(device)


def to_bits(t: torch.Tensor) -> np.ndarray:
    """Device bf16/int16 tensor -> uint16 numpy bits."""
    if t.dtype == torch.bfloat16:
        t = t.view(torch.int16)
    return t.cpu().numpy().view(np.uint16)


def bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


class DeviceWorkload:
    """Uploads a :class:`Workload` and registers its pool with the library."""

    def __init__(self, wl: Workload, device: str = "cuda:0", replicas: int = 1):
        """``replicas`` > 1 uploads that many copies of the K/V pool (same
        contents, own addresses), each registered as its own pool: a benchmark
        rotates calls over them so that a working set smaller than the GPU's
        caches is still read from HBM."""
        self.wl = wl
        self.cfg = wl.cfg
        self.device = torch.device(device)
        c = wl.cfg
        self.hq, self.hkv, self.d = c.hq, c.hkv, c.head_dim
        self.scale = 1.0 / math.sqrt(c.head_dim)
        self.k_pool = _dev16(wl.k_pool, self.device)
        self.v_pool = _dev16(wl.v_pool, self.device)
        self.k_pools = [self.k_pool] + [self.k_pool.clone() for _ in range(replicas - 1)]
        self.v_pools = [self.v_pool] + [self.v_pool.clone() for _ in range(replicas - 1)]
        self.pools = [mw.mw_kv_pool_create(wl.num_pages, c.page_size, c.hkv, c.head_dim, k.data_ptr(), v.data_ptr())
                      for k, v in zip(self.k_pools, self.v_pools)]
        self.pool = self.pools[0]
        self.pre_bt = _dev32(wl.pre_bt[None, :], self.device)
        self.dec_bt = _dev32(wl.dec_bt, self.device)
        self.dec_lens = wl.dec_lens.astype(np.int32)
        self.d_dec_lens = _dev32(self.dec_lens, self.device)
        self.q_pre = _dev16(wl.q_pre, self.device)
        self.q_dec = _dev16(wl.q_dec, self.device)
        self.o_pre = torch.zeros_like(self.q_pre)
        self.o_dec = torch.zeros_like(self.q_dec)
        self._ws = {}
        self._pre_ws = None
        self._pre_args = {}
        self._dec_start = None

    @property
    def replicas(self) -> int:
        return len(self.pools)

    def close(self):
        for p in self.pools:
            mw.mw_kv_pool_destroy(p)
        self.pools = []
        self.pool = None

    # ----------------------------------------------------------- prefill --
    def _prefill_args(self, r: int, n: int):
        key = (r, n)
        if key not in self._pre_args:
            self._pre_args[key] = (_dev32([0, n], self.device), _dev32([r], self.device))
        return self._pre_args[key]

    def prefill_workspace(self) -> torch.Tensor:
        """Workspace for the key-range split of any of the workload's prefill
        chunks on any stream (the split is used only where the launch would
        leave CUs idle)."""
        if self._pre_ws is None:
            nbytes = max([mw.mw_prefill_workspace_size(self.hq, self.hkv, self.d, [n], [r])
                          for r, n in self.cfg.pre_chunks] + [16])
            self._pre_ws = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        return self._pre_ws

    def prefill(self, r: int, n: int, stream=0, timing=None, out: Optional[torch.Tensor] = None,
                split: bool = True):
        """Causal prefill of positions [r, r+n) over prefix r; returns the
        output rows [n][Hq][D] (a view of ``out`` or of the workload's buffer).
        split=False: the plain call, without the key-range split."""
        indptr, pref = self._prefill_args(r, n)
        q = self.q_pre[r:r + n]
        o = self.o_pre[r:r + n] if out is None else out
        if split:
            ws = self.prefill_workspace()
            mw.mw_prefill_attn_ws(self.pool, self.hq, self.hkv, self.d, self.scale, [n], [r],
                                  indptr.data_ptr(), pref.data_ptr(), self.pre_bt.data_ptr(),
                                  self.pre_bt.shape[1], q.data_ptr(), o.data_ptr(), ws.data_ptr(),
                                  ws.numel(), stream, timing)
        else:
            mw.mw_prefill_attn(self.pool, self.hq, self.hkv, self.d, self.scale, [n], [r],
                               indptr.data_ptr(), pref.data_ptr(), self.pre_bt.data_ptr(),
                               self.pre_bt.shape[1], q.data_ptr(), o.data_ptr(), stream, timing)
        return o

    def write_prefill_kv(self, r: int, n: int, k_new: torch.Tensor, v_new: torch.Tensor,
                         stream=0, timing=None):
        indptr, pref = self._prefill_args(r, n)
        mw.mw_kv_pool_write(self.pool, [n], [r], indptr.data_ptr(), pref.data_ptr(),
                            self.pre_bt.data_ptr(), self.pre_bt.shape[1], k_new.data_ptr(),
                            v_new.data_ptr(), stream, timing)

    # ------------------------------------------------------------ decode --
    def workspace(self, chunk_pages: int = 0) -> torch.Tensor:
        if chunk_pages not in self._ws:
            nbytes = mw.mw_decode_workspace_size(self.hq, self.hkv, self.d, self.dec_lens,
                                                 chunk_pages)
            self._ws[chunk_pages] = torch.empty(max(nbytes, 16), dtype=torch.uint8,
                                                device=self.device)
        return self._ws[chunk_pages]

    def decode(self, stream=0, timing=None, chunk_pages: int = 0,
               out: Optional[torch.Tensor] = None, replica: int = 0):
        ws = self.workspace(chunk_pages)
        o = self.o_dec if out is None else out
        mw.mw_decode_attn(self.pools[replica], self.hq, self.hkv, self.d, self.scale, self.dec_lens,
                          self.d_dec_lens.data_ptr(), self.dec_bt.data_ptr(), self.dec_bt.shape[1],
                          self.q_dec.data_ptr(), o.data_ptr(), ws.data_ptr(), ws.numel(),
                          chunk_pages, stream, timing)
        return o

    def write_decode_kv(self, k_new: torch.Tensor, v_new: torch.Tensor, stream=0, timing=None,
                        replica: int = 0):
        """Appends each decode sequence's newest token at position L-1."""
        B = len(self.dec_lens)
        if self._dec_start is None:
            self._dec_start = (_dev32(np.arange(B + 1), self.device),
                               _dev32(self.dec_lens - 1, self.device))
        indptr, start = self._dec_start
        mw.mw_kv_pool_write(self.pools[replica], np.ones(B, np.int32), self.dec_lens - 1,
                            indptr.data_ptr(), start.data_ptr(), self.dec_bt.data_ptr(),
                            self.dec_bt.shape[1], k_new.data_ptr(), v_new.data_ptr(), stream,
                            timing)


    # ------------------------------------------------------------ engine --
    def engine_args(self, chunk_pages: int = 0):
        """(decode, prefill) argument dicts for :func:`mw.mw_engine_run`: one
        decode call over every sequence, and one prefill call whose batch holds
        every prefill chunk (chunk j attends to its prefix and causally to
        itself, so the batch equals running the chunks in order)."""
        c = self.cfg
        chunks = list(c.pre_chunks)
        for (r0, n0), (r1, _) in zip(chunks, chunks[1:]):
            if r1 != r0 + n0:
                raise ValueError("prefill chunks must be contiguous")
        if "engine" not in self._pre_args:
            indptr = np.concatenate([[0], np.cumsum([n for _, n in chunks])])
            bt = np.repeat(self.wl.pre_bt[None, :], len(chunks), axis=0)
            self._pre_args["engine"] = (_dev32(indptr, self.device), _dev32([r for r, _ in chunks], self.device),
                                        _dev32(bt, self.device))
        indptr, pref, bt = self._pre_args["engine"]
        r0 = chunks[0][0]
        ws = self.workspace(chunk_pages)
        shape = dict(hq=self.hq, hkv=self.hkv, head_dim=self.d, scale=self.scale)
        dec = dict(pool=self.pool, seq_lens=self.dec_lens, d_seq_lens=self.d_dec_lens.data_ptr(),
                   d_block_table=self.dec_bt.data_ptr(), bt_stride=self.dec_bt.shape[1],
                   d_q=self.q_dec.data_ptr(), d_out=self.o_dec.data_ptr(), d_workspace=ws.data_ptr(),
                   workspace_bytes=ws.numel(), chunk_pages=chunk_pages, **shape)
        pre = dict(pool=self.pool, new_lens=[n for _, n in chunks], prefix_lens=[r for r, _ in chunks],
                   d_qo_indptr=indptr.data_ptr(), d_prefix_lens=pref.data_ptr(), d_block_table=bt.data_ptr(),
                   bt_stride=bt.shape[1], d_q=self.q_pre[r0].data_ptr(), d_out=self.o_pre[r0].data_ptr(), **shape)
        return dec, pre


class Timing:
    """Owns an mw_timing handle."""

    def __init__(self):
        self.h = mw.mw_timing_create()

    def close(self):
        if self.h is not None:
            mw.mw_timing_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def elapsed(self) -> Tuple[float, float]:
        return mw.mw_timing_elapsed(self.h)

    def kernel_ms(self, k: int) -> float:
        return mw.mw_timing_kernel_ms(self.h, k)

    def kernels(self) -> int:
        return mw.mw_timing_kernels(self.h)

    def all_kernels_ms(self) -> float:
        """GPU time of every kernel of the call (a split prefill has two)."""
        return sum(self.kernel_ms(k) for k in range(self.kernels()))


class Partition:
    """Owns an mw_partition; exposes its streams as torch ExternalStreams."""

    def __init__(self, prefill_cus: int, decode_cus: int, device: int = 0):
        self.h = mw.mw_partition_create(device, prefill_cus, decode_cus)
        self.prefill_stream, self.decode_stream = mw.mw_partition_streams(self.h)
        self.prefill_cus, self.decode_cus = prefill_cus, decode_cus

    def torch_streams(self):
        return (torch.cuda.ExternalStream(self.prefill_stream),
                torch.cuda.ExternalStream(self.decode_stream))

    def masks(self):
        return mw.mw_partition_masks(self.h)

    def close(self):
        if self.h is not None:
            mw.mw_partition_destroy(self.h)
            self.h = None
