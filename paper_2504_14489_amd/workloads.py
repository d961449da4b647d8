"""Seeded synthetic inputs for paged prefill/decode attention.

This module is the only code shared by the CPU oracle's tests and the HIP
path's tests and benchmark.  It draws random numbers, rounds them to bf16 and
lays them out as a paged K/V pool with block tables.  It contains none of the
attention arithmetic.

Workload shapes follow the serving mixes the paper characterises (Sec. 2.1,
Table "tb:tasks"; Sec. 2.2: a 2K-token prefill chunk next to a decode batch of
32) at the attention-layer shapes of Llama-3-8B / 70B (32 or 64 query heads,
8 KV heads, head_dim 128) with 16-token pages.

Layout produced (all bf16 values are carried as raw ``uint16`` bit patterns):

* ``k_pool``, ``v_pool``: ``[P][Hkv][S][D]`` - one (page, kv-head) block is
  ``S*D`` contiguous elements.  Page ``P-1`` is a dedicated NaN page that
  block-table padding points to.
* prefill block table ``pre_bt``: ``[max_pre_pages]`` int32.
* decode block tables ``dec_bt``: ``[B][dec_bt_stride]`` int32, padded with the
  NaN page.

Poison (so that a kernel reading what it must not read fails parity):

* never-allocated pages hold bf16 NaN;
* slots past a sequence's last token inside its last page hold a large finite
  value (a masked-out key contributes ``exp(-inf) * finite = 0``; an unmasked
  one dominates the softmax).

Draw order from ``numpy.random.Generator(PCG64(seed))``: decode lengths, page
permutation, prefill Q, decode Q.  K and V are drawn per block of 1024 pages,
block j of K from ``PCG64(SeedSequence([seed, 1, j]))`` and of V from
``PCG64(SeedSequence([seed, 2, j]))``, so that blocks can be drawn in
parallel.
"""
from __future__ import annotations

import concurrent.futures
import dataclasses
import math
import os
from typing import List, Optional, Tuple

import numpy as np

PAGE_SIZE = 16
HEAD_DIM = 128
BF16_NAN = 0x7FC0
BF16_POS_INF = 0x7F80
BF16_NEG_INF = 0xFF80
# 29952.0 in bf16 (0x46EA): finite, and large enough that an unmasked slack key
# would dominate every softmax row it leaks into.
BF16_SLACK_POISON = 0x46EA


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 with round-to-nearest-even; return uint16 bits."""
    x = np.asarray(x, dtype=np.float32)
    if not x.flags.c_contiguous:
        x = np.ascontiguousarray(x)
    out = np.empty(x.shape, dtype=np.uint16)
    flat_x = x.reshape(-1)
    flat_o = out.reshape(-1)
    step = 1 << 24
    for i in range(0, flat_x.size, step):
        u = flat_x[i:i + step].view(np.uint32)
        r = (u >> 16) & np.uint32(1)
        r += np.uint32(0x7FFF)
        r += u                      # finite values cannot overflow 32 bits
        r >>= 16
        flat_o[i:i + step] = r
        nan = np.isnan(flat_x[i:i + step])
        if nan.any():
            flat_o[i:i + step][nan] = BF16_NAN
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass(frozen=True)
class Config:
    """One synthetic workload: a prefill sequence next to a decode batch."""
    name: str
    hq: int
    hkv: int
    # prefill: list of (prefix_len r, new_len n) calls over ONE sequence whose
    # K/V for positions [0, r_last + n_last) is resident in the pool.
    pre_chunks: Tuple[Tuple[int, int], ...]
    dec_batch: int
    dec_len_dist: str            # "uniform" | "lognormal"
    dec_len_lo: int
    dec_len_hi: int
    pool_pages: Optional[int]    # None = sized to fit exactly
    prefill_cus: Tuple[int, ...]
    decode_cus: Tuple[int, ...]
    seed: int = 0
    head_dim: int = HEAD_DIM
    page_size: int = PAGE_SIZE
    lognormal_median: float = 2048.0
    lognormal_sigma: float = 0.8

    @property
    def pre_total(self) -> int:
        return max(r + n for r, n in self.pre_chunks) if self.pre_chunks else 0


# The five workloads, by what they are.
CONFIGS = {
    # tiny single layer; 8 q-heads / 2 kv-heads; 256-page pool; 50/50 split
    "tiny": Config("tiny", 8, 2, ((0, 256),), 4, "uniform", 128, 512, 256,
                   (128,), (128,)),
    # Llama-3-8B-shaped layer: 2048-token chunk, 64 decodes in [512, 4096]
    "llama8b": Config("llama8b", 32, 8, ((0, 2048),), 64, "uniform", 512, 4096,
                      None, (64,), (192,)),
    # Llama-3-70B-shaped layer: 8192 tokens in four 2048 chunks; 128 decodes
    # with lognormal contexts (median 2048, sigma 0.8, clipped to [64, 16384])
    "llama70b": Config("llama70b", 64, 8,
                       ((0, 2048), (2048, 2048), (4096, 2048), (6144, 2048)),
                       128, "lognormal", 64, 16384, None, (96,), (160,)),
    # one GPU's shard of the Llama-3-70B layer at tensor-parallel degree 8
    # (8 q-heads / 1 kv-head per GPU), same tokens and decode batch as llama70b
    "llama70b_tp8": Config("llama70b_tp8", 8, 1,
                           ((0, 2048), (2048, 2048), (4096, 2048), (6144, 2048)),
                           128, "lognormal", 64, 16384, None, (96,), (160,)),
    # long context 8B: 4096 new tokens over a 28672-token cached prefix;
    # 32 decodes in [16384, 32768]
    "longctx8b": Config("longctx8b", 32, 8, ((28672, 4096),), 32, "uniform",
                        16384, 32768, None, (128,), (128,)),
    # CU-partition sweep, 8B shapes: 4096-token prefill, 256 decodes in
    # [1024, 8192]; prefill CUs swept over multiples of 32
    "sweep8b": Config("sweep8b", 32, 8, ((0, 4096),), 256, "uniform", 1024, 8192,
                      None, (32, 64, 96, 128, 160, 192, 224),
                      (224, 192, 160, 128, 96, 64, 32)),
}


def custom_config(name="custom", hq=4, hkv=2, pre_chunks=((0, 33),), dec_batch=3,
                  dec_len_lo=1, dec_len_hi=40, dec_len_dist="uniform",
                  pool_pages=None, seed=0, head_dim=HEAD_DIM,
                  page_size=PAGE_SIZE) -> Config:
    """A small configuration for tests (ragged lengths, odd sizes)."""
    return Config(name, hq, hkv, tuple(tuple(c) for c in pre_chunks), dec_batch,
                  dec_len_dist, dec_len_lo, dec_len_hi, pool_pages, (0,), (0,),
                  seed=seed, head_dim=head_dim, page_size=page_size)


@dataclasses.dataclass
class Workload:
    cfg: Config
    k_pool: np.ndarray        # uint16 [P][Hkv][S][D]
    v_pool: np.ndarray        # uint16 [P][Hkv][S][D]
    nan_page: int
    pre_len: int              # tokens of the prefill sequence resident in the pool
    pre_bt: np.ndarray        # int32 [pre_bt_stride]
    q_pre: np.ndarray         # uint16 [pre_len][Hq][D] (rows for every position)
    dec_lens: np.ndarray      # int32 [B]
    dec_bt: np.ndarray        # int32 [B][dec_bt_stride]
    q_dec: np.ndarray         # uint16 [B][Hq][D]
    perm: np.ndarray          # int32 [P-1] page permutation used for dealing

    @property
    def num_pages(self) -> int:
        return self.k_pool.shape[0]

    # ---- logical (unpaged) views, used only by tests -----------------------
    def logical_kv(self, bt: np.ndarray, length: int) -> Tuple[np.ndarray, np.ndarray]:
        """Gather tokens [0, length) of a sequence: uint16 [length][Hkv][D] each."""
        S = self.cfg.page_size
        t = np.arange(length)
        pages = bt[t // S]
        slots = t % S
        k = self.k_pool[pages, :, slots, :]
        v = self.v_pool[pages, :, slots, :]
        return np.ascontiguousarray(k), np.ascontiguousarray(v)

    def pre_new_kv(self, r: int, n: int) -> Tuple[np.ndarray, np.ndarray]:
        """K/V rows of prefill positions [r, r+n): uint16 [n][Hkv][D] each."""
        k, v = self.logical_kv(self.pre_bt, r + n)
        return np.ascontiguousarray(k[r:]), np.ascontiguousarray(v[r:])

    def dec_new_kv(self) -> Tuple[np.ndarray, np.ndarray]:
        """K/V of each decode sequence's newest token (position L-1): [B][Hkv][D]."""
        ks, vs = [], []
        for b, L in enumerate(self.dec_lens):
            k, v = self.logical_kv(self.dec_bt[b], int(L))
            ks.append(k[-1])
            vs.append(v[-1])
        return np.stack(ks), np.stack(vs)


def draw_decode_lengths(cfg: Config, rng: np.random.Generator) -> np.ndarray:
    if cfg.dec_batch == 0:
        return np.zeros(0, dtype=np.int32)
    if cfg.dec_len_dist == "uniform":
        L = rng.integers(cfg.dec_len_lo, cfg.dec_len_hi + 1, size=cfg.dec_batch)
    elif cfg.dec_len_dist == "lognormal":
        x = rng.normal(math.log(cfg.lognormal_median), cfg.lognormal_sigma,
                       size=cfg.dec_batch)
        L = np.clip(np.rint(np.exp(x)), cfg.dec_len_lo, cfg.dec_len_hi)
    else:
        raise ValueError(cfg.dec_len_dist)
    return L.astype(np.int32)


_PAGE_BLOCK = 1024


def _pool_bf16(seed: int, stream: int, shape) -> np.ndarray:
    """N(0,1) bf16 pool [P][...]: page block j from its own seeded stream."""
    P = shape[0]
    out = np.empty(shape, dtype=np.uint16)

    def fill(j):
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream, j])))
        lo, hi = j * _PAGE_BLOCK, min(P, (j + 1) * _PAGE_BLOCK)
        x = g.standard_normal(size=(hi - lo,) + tuple(shape[1:]), dtype=np.float32)
        out[lo:hi] = f32_to_bf16_bits(x)

    blocks = range(-(-P // _PAGE_BLOCK))
    workers = max(1, min(16, os.cpu_count() or 1))
    with concurrent.futures.ThreadPoolExecutor(workers) as ex:
        list(ex.map(fill, blocks))
    return out


def _normal_bf16(rng: np.random.Generator, shape, scale: float = 1.0) -> np.ndarray:
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if scale != 1.0:
        x *= np.float32(scale)
    return f32_to_bf16_bits(x)


def make_workload(cfg: Config, seed: Optional[int] = None, q_scale: float = 1.0,
                  dec_lens: Optional[np.ndarray] = None,
                  slack_bits: Tuple[int, int] = (BF16_SLACK_POISON, BF16_SLACK_POISON)) -> Workload:
    """Build the pool image, block tables and queries for ``cfg``.

    ``q_scale`` multiplies Q before rounding (a "peaked" variant that makes
    the running softmax maximum move).  ``dec_lens`` overrides the drawn decode
    lengths (the draw still happens, keeping the stream order fixed).
    ``slack_bits`` are the bf16 patterns written to the K and V slots past each
    sequence's end in its last page (default: the large finite poison; tests
    also use NaN and Inf there, which no correct kernel lets into a result).
    """
    seed = cfg.seed if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(seed))
    S, D, Hkv, Hq = cfg.page_size, cfg.head_dim, cfg.hkv, cfg.hq
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")

    lens = draw_decode_lengths(cfg, rng)
    if dec_lens is not None:
        lens = np.asarray(dec_lens, dtype=np.int32)
    B = len(lens)
    pre_len = cfg.pre_total
    pre_pages = -(-pre_len // S)
    dec_pages = [-(-int(L) // S) for L in lens]
    need = pre_pages + sum(dec_pages)
    data_pages = need if cfg.pool_pages is None else cfg.pool_pages
    if data_pages < need:
        raise ValueError(f"pool of {data_pages} pages cannot hold {need}")
    P = data_pages + 1            # + the dedicated NaN page
    nan_page = P - 1

    perm = rng.permutation(data_pages).astype(np.int32)
    cursor = 0
    pre_bt = perm[cursor:cursor + pre_pages].copy()
    cursor += pre_pages
    dec_stride = max(dec_pages) if dec_pages else 1
    dec_bt = np.full((B, max(dec_stride, 1)), nan_page, dtype=np.int32)
    for b, np_b in enumerate(dec_pages):
        dec_bt[b, :np_b] = perm[cursor:cursor + np_b]
        cursor += np_b
    if pre_pages == 0:
        pre_bt = np.full(1, nan_page, dtype=np.int32)

    q_pre = _normal_bf16(rng, (pre_len, Hq, D), q_scale)
    q_dec = _normal_bf16(rng, (B, Hq, D), q_scale)
    k_pool = _pool_bf16(seed, 1, (P, Hkv, S, D))
    v_pool = _pool_bf16(seed, 2, (P, Hkv, S, D))

    # poison: every page not dealt to a sequence is NaN (incl. the NaN page)
    used = np.zeros(P, dtype=bool)
    used[pre_bt[:pre_pages]] = True
    for b, np_b in enumerate(dec_pages):
        used[dec_bt[b, :np_b]] = True
    k_pool[~used] = BF16_NAN
    v_pool[~used] = BF16_NAN
    # slack slots past the end of each sequence's last page
    def poison_tail(bt_row, length):
        if length % S:
            last = bt_row[length // S]
            k_pool[last, :, length % S:, :] = slack_bits[0]
            v_pool[last, :, length % S:, :] = slack_bits[1]
    if pre_len:
        poison_tail(pre_bt, pre_len)
    for b, L in enumerate(lens):
        poison_tail(dec_bt[b], int(L))

    return Workload(cfg=cfg, k_pool=k_pool, v_pool=v_pool, nan_page=nan_page,
                    pre_len=pre_len, pre_bt=pre_bt, q_pre=q_pre, dec_lens=lens,
                    dec_bt=dec_bt, q_dec=q_dec, perm=perm)
