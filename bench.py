#!/usr/bin/env python3
"""Benchmark: paged GQA prefill + decode attention multiplexed on split CUs.

One step = one pass of the whole hot path over one batch of synthetic input,
with the two phases on disjoint CU partitions of the GPU (decode enqueued
first, as the paper launches the decode iteration before prefill, Sec. 3.2.2):

  decode stream : m x (append each sequence's new K/V, decode attention:
                  one kernel, the balanced split, whose last work-group on
                  each (sequence, kv head) merges that segment's pieces)
  prefill stream: append each chunk's new K/V, causal prefill attention

m is the number of decode iterations that fit in one prefill call when the
two run side by side (at least 1; from the warm-up of the multiplexed loop),
so both partitions stay busy for the whole timed region, as in the paper's
bubble-less multiplexing.

The default run measures every workload in turn (tiny as a parity case, the
8B- and 70B-shaped layers, one GPU's tensor-parallel-8 shard of the 70B layer,
the CU-partition sweep with its contention table, and the long-context 8B
layer, which carries the headline: the largest single-GPU workload).  For each:

* isolated per-call latency of each phase on its own CUs, with the L2 and
  Infinity Cache flushed before every timed call (512 MiB read on the same
  stream), and on the whole GPU; K/V pool replicas rotated per decode call
  when the decode working set is under 512 MB, so it is read from HBM;
* the multiplexed timed region (per-kernel HIP events on each kernel's own
  stream), the contention slowdown and whether multiplexed outputs equal the
  isolated ones bit for bit;
* the roofline of each kernel against the published peaks, the pro-rata
  share of its CUs, the measured MFMA ceiling (prefill) or stream-read
  ceiling (decode) of the same CUs;
* the same step without partitions (serial, free streams, one fused launch);
* parity of the multiplexed outputs with the CPU oracle (every decode
  sequence; each prefill chunk's rows at the edges of every 16-row group of
  every query block), whose timings are the CPU baseline of that workload.

Printed: one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import platform
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "prefill attn TFLOP/s + decode attn HBM GB/s, multiplexed on split CUs"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
BF16_PEAK_TFLOPS = 2516.6      # MI355X dense bf16 MFMA (256 CUs x 4096 flop/clk x 2.4 GHz)
N_CU = 256
ORDER = ["tiny", "llama8b", "llama70b", "llama70b_tp8", "sweep8b", "longctx8b"]
HEADLINE = "longctx8b"         # the largest workload that fits one GPU
PARITY_ONLY = {"tiny"}         # ~1 us of work: launch latency, not the kernels, sets its time
FLUSH_BYTES = 512 << 20        # > 2 x the 256 MiB Infinity Cache
REPLICA_BELOW = 512e6          # decode K/V bytes below which pool replicas rotate
REPLICA_CYCLE = 768e6          # bytes the rotation cycles through
MARK_BASE = 4096               # trace-mark ids: MARK_BASE + 64 * workload + 2 * partition + (0 start, 1 end)

DESC = {
    "tiny": "tiny layer: 8 q-heads/2 kv-heads, 256-token prefill, 4 decodes U[128,512]",
    "llama8b": "Llama-3-8B-shaped attention layer: 32 q-heads/8 kv-heads, d=128, 16-token pages; "
               "2048-token prefill chunk (no prefix) + 64 decodes with contexts U[512,4096]",
    "llama70b": "Llama-3-70B-shaped attention layer: 64 q-heads/8 kv-heads; 8192-token prefill in "
                "four 2048-token chunks + 128 decodes, lognormal contexts (median 2048, sigma 0.8)",
    "llama70b_tp8": "one GPU's tensor-parallel-8 shard of the Llama-3-70B attention layer: 8 q-heads/1 kv-head; "
                    "8192-token prefill in four 2048-token chunks + 128 decodes, lognormal contexts",
    "longctx8b": "Long-context 8B-shaped attention layer: 32 q-heads/8 kv-heads, d=128, 16-token pages; "
                 "4096 new tokens over a 28672-token cached prefix + 32 decodes with contexts U[16384,32768]",
    "sweep8b": "8B shapes: 4096-token prefill + 256 decodes U[1024,8192], prefill CUs swept over 32..224",
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--configs", default=",".join(ORDER),
                    help="comma-separated workloads to measure: " + ", ".join(ORDER))
    ap.add_argument("--config", default="",
                    help="measure this one workload only (it then carries the headline)")
    ap.add_argument("--partition", type=int, default=-1,
                    help="index into each workload's CU splits (sweep8b has 7); -1 = all")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--iso-reps", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle (parity and CPU baseline)")
    ap.add_argument("--table", default="", help="also write the per-workload and sweep tables (Markdown) here")
    ap.add_argument("--traffic-pass", action="store_true",
                    help="run each kernel of --config once on its partition plus a device copy of known size "
                         "(the command profiled by rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE), then exit")
    a = ap.parse_args()
    a.names = [a.config] if a.config else [n for n in a.configs.split(",") if n]
    for n in a.names:
        if n not in ORDER:
            ap.error(f"unknown workload {n!r}")
    a.headline = HEADLINE if HEADLINE in a.names else a.names[-1]
    return a


def median(x):
    return statistics.median(x) if x else float("nan")


def p90(x):
    return float(np.percentile(x, 90)) if x else float("nan")


class Device:
    """What every workload's measurement shares: the whole-GPU streams, the
    flush buffer and the probe buffers."""

    def __init__(self):
        import torch
        self.torch = torch
        self.dev = torch.device("cuda:0")
        self.full = torch.cuda.Stream()            # no CU mask: the whole GPU
        self.full2 = torch.cuda.Stream()
        self.flush_buf = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device=self.dev)
        self.read_buf = torch.empty(1 << 30, dtype=torch.uint8, device=self.dev)
        self.sink = torch.empty(1 << 16, dtype=torch.int32, device=self.dev)
        self.fsink = torch.empty(1 << 16, dtype=torch.float32, device=self.dev)
        torch.cuda.synchronize()
        self._ceilings = {}

    def flush(self, stream):
        from paper_2504_14489_amd import mw
        mw.mw_cache_flush(self.flush_buf.data_ptr(), FLUSH_BYTES, stream)

    def stream_ceiling(self, stream, n_cus, reps=5):
        """HBM read rate the CUs of `stream` reach on a plain 1 GiB stream (GB/s)."""
        from paper_2504_14489_amd import mw
        from paper_2504_14489_amd.device import Timing
        ts = [Timing() for _ in range(reps + 1)]
        self.torch.cuda.synchronize()
        for t in ts:
            mw.mw_stream_read(self.read_buf.data_ptr(), self.read_buf.numel(), self.sink.data_ptr(), 8 * n_cus,
                              stream, t.h)
        self.torch.cuda.synchronize()
        ms = median([t.kernel_ms(0) for t in ts[1:]])
        return self.read_buf.numel() / (ms * 1e-3) / 1e9

    def mfma_ceiling(self, stream, n_cus, reps=3):
        """bf16 matrix-core rate the CUs of `stream` sustain (TFLOP/s): four
        256-thread work-groups per CU issuing MFMAs from registers."""
        from paper_2504_14489_amd import mw
        from paper_2504_14489_amd.device import Timing
        ts = [Timing() for _ in range(reps + 1)]
        self.torch.cuda.synchronize()
        flop = 0.0
        for t in ts:
            flop = mw.mw_mfma_peak(4 * n_cus, 4096, self.fsink.data_ptr(), stream, t.h)
        self.torch.cuda.synchronize()
        ms = min(t.kernel_ms(0) for t in ts[1:])
        return flop / (ms * 1e-3) / 1e12


class Bench:
    """One workload resident on the GPU and its measurements."""

    def __init__(self, name, args, gpu: Device, index: int):
        from paper_2504_14489_amd import accounting, workloads as W
        from paper_2504_14489_amd.device import DeviceWorkload, Partition, Timing, _dev16

        self.torch = gpu.torch
        self.gpu = gpu
        self.Timing = Timing
        self.Partition = Partition
        self.args = args
        self.index = index
        self.cfg = W.CONFIGS[name]
        c = self.cfg
        t = time.time()
        self.wl = W.make_workload(c, seed=args.seed)
        self.chunks = list(c.pre_chunks)
        self.pre_flop = accounting.prefill_flops(c.hq, c.head_dim, self.chunks)
        self.dec_bytes = accounting.decode_bytes(c.hq, c.hkv, c.head_dim, self.wl.dec_lens)
        kv = 4 * c.hkv * c.head_dim * int(np.sum(self.wl.dec_lens, dtype=np.int64))
        self.replicas = 1 if kv >= REPLICA_BELOW else int(min(64, max(2, math.ceil(REPLICA_CYCLE / kv))))
        self.dw = DeviceWorkload(self.wl, replicas=self.replicas)
        log(f"[bench] {name}: {self.wl.num_pages} pages, {len(self.wl.dec_lens)} decodes, decode K/V "
            f"{kv / 1e6:.1f} MB x {self.replicas} pool cop{'y' if self.replicas == 1 else 'ies'}, "
            f"ready in {time.time() - t:.1f}s")
        # the step's appended K/V rows (bit-identical to what the pool holds)
        self.pre_new = [tuple(_dev16(a, self.dw.device) for a in self.wl.pre_new_kv(r, n))
                        for r, n in self.chunks]
        kd, vd = self.wl.dec_new_kv()
        self.dec_new = (_dev16(kd, self.dw.device), _dev16(vd, self.dw.device))
        self._rep = 0
        self.torch.cuda.synchronize()

    # ------------------------------------------------------------ phases --
    def prefill_call(self, stream, tp=None):
        """All prefill chunks of the step: append, then attention (on the first
        pool copy; the prefill's own K/V is small and re-read by design)."""
        for (r, n), (k, v) in zip(self.chunks, self.pre_new):
            self.dw.write_prefill_kv(r, n, k, v, stream)
            self.dw.prefill(r, n, stream, tp.h if tp else None)

    def decode_call(self, stream, td=None):
        """One decode iteration (append + attention) on the next pool copy."""
        rep = self._rep % self.replicas
        self._rep += 1
        self.dw.write_decode_kv(self.dec_new[0], self.dec_new[1], stream, None, replica=rep)
        self.dw.decode(stream, td.h if td else None, replica=rep)

    # ---------------------------------------------------------- isolated --
    def isolated(self, which, stream, reps):
        """Per-call kernel times of one phase alone on `stream`, the caches
        flushed (untimed, same stream) before every call."""
        torch = self.torch
        nchunk = len(self.chunks) if which == "prefill" else 1
        tks = [[self.Timing() for _ in range(nchunk)] for _ in range(reps)]
        torch.cuda.synchronize()
        for i in range(reps):
            if which == "prefill":
                for (r, n), (k, v), tk in zip(self.chunks, self.pre_new, tks[i]):
                    self.dw.write_prefill_kv(r, n, k, v, stream)
                    self.gpu.flush(stream)
                    self.dw.prefill(r, n, stream, tk.h)
            else:
                rep = self._rep % self.replicas
                self._rep += 1
                self.dw.write_decode_kv(self.dec_new[0], self.dec_new[1], stream, None, replica=rep)
                self.gpu.flush(stream)
                self.dw.decode(stream, tks[i][0].h, replica=rep)
        torch.cuda.synchronize()
        out = {"k0": [sum(tk.all_kernels_ms() if which == "prefill" else tk.kernel_ms(0) for tk in row)
                      for row in tks],
               "kernels": tks[-1][0].kernels(),
               "call": [sum(tk.elapsed()[0] for tk in row) for row in tks]}
        if which == "decode" and out["kernels"] > 1:
            out["k1"] = [row[0].kernel_ms(1) for row in tks]
        return out

    # ------------------------------------------------------- multiplexed --
    def multiplexed(self, part, steps, m, mark=None):
        from paper_2504_14489_amd import mw
        torch = self.torch
        ps, ds = part.prefill_stream, part.decode_stream
        tp = [[self.Timing() for _ in self.chunks] for _ in range(steps)]
        td = [[self.Timing() for _ in range(m)] for _ in range(steps)]
        if mark is not None:
            mw.mw_trace_mark(mark, ds)
            mw.mw_trace_mark(mark, ps)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(steps):
            for j in range(m):                      # decode first
                self.decode_call(ds, td[k][j])
            for (r, n), (kk, vv), t in zip(self.chunks, self.pre_new, tp[k]):
                self.dw.write_prefill_kv(r, n, kk, vv, ps)
                self.dw.prefill(r, n, ps, t.h)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        if mark is not None:
            mw.mw_trace_mark(mark + 1, ds)
            mw.mw_trace_mark(mark + 1, ps)
            torch.cuda.synchronize()
        ref = td[0][0].h
        return {"wall_s": wall,
                "prefill_k": [sum(t.all_kernels_ms() for t in tp[k]) for k in range(steps)],
                "prefill_kernels": tp[0][0].kernels(),
                "decode_k0": [t.kernel_ms(0) for k in range(steps) for t in td[k]],
                "decode_call": [t.elapsed()[0] for k in range(steps) for t in td[k]],
                "prefill_window_ms": [min(mw.mw_timing_offsets(tp[k][0].h, ref)[0] for k in range(steps)),
                                      max(mw.mw_timing_offsets(tp[k][-1].h, ref)[1] for k in range(steps))],
                "decode_window_ms": [0.0, mw.mw_timing_offsets(td[-1][-1].h, ref)[1]]}

    # --------------------------------------------- temporal baselines --
    def temporal(self, kind, steps, m):
        """Wall ms per step of the same work without CU partitions, on the
        whole GPU: "serial" = prefill, then m decode iterations, one stream;
        "free" = the two phases on two unmasked streams (the hardware shares
        the CUs); "fused" = appends, one fused prefill + decode launch, then
        m - 1 more decode iterations."""
        from paper_2504_14489_amd import mw
        torch = self.torch
        s1, s2 = self.gpu.full.cuda_stream, self.gpu.full2.cuda_stream
        if not hasattr(self, "eng_dec"):
            self.eng_dec, self.eng_pre = self.dw.engine_args()
        td = []

        def step(timed=False):
            if kind == "serial":
                self.prefill_call(s1)
                for _ in range(m):
                    self.decode_call(s1)
            elif kind == "free":
                for _ in range(m):
                    t = self.Timing() if timed else None
                    self.decode_call(s2, t)
                    if t is not None:
                        td.append(t)
                self.prefill_call(s1)
            else:
                for (r, n), (k, v) in zip(self.chunks, self.pre_new):
                    self.dw.write_prefill_kv(r, n, k, v, s1)
                self.dw.write_decode_kv(self.dec_new[0], self.dec_new[1], s1)
                mw.mw_fused_attn(self.eng_pre, self.eng_dec, s1)
                for _ in range(m - 1):
                    self.decode_call(s1)

        for _ in range(max(1, self.args.warmup)):
            step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            step(timed=True)
        torch.cuda.synchronize()
        ms = 1e3 * (time.perf_counter() - t0) / steps
        # a decode token is ready when its iteration ends: on one stream that
        # is the end of the step, next to the prefill it is the decode call
        dec_ms = median([t.elapsed()[0] for t in td]) if td else ms / m
        return ms, dec_ms

    def close(self):
        self.dw.close()


# ------------------------------------------------------------- rooflines --
KERNEL_SOURCES = {"k_prefill_attn": ("prefill_attn.hip", "prefill_block.h"),
                  "k_decode_balanced": ("decode_attn.hip", "decode_block.h")}


def source_sha(kernel):
    """Hash of the kernel's sources (launcher and work-group body)."""
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kernel]:
        h.update(open(os.path.join(ROOT, "paper_2504_14489_amd", "csrc", name), "rb").read())
    return h.hexdigest()[:16]


def committed_traffic(kernel, workload):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE/WRITE_SIZE
    summary, scaled by the copy-kernel calibration it records; None when the
    summary is missing or the kernel's source has changed since."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.txt")
    if kernel not in KERNEL_SOURCES or not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get(f"{kernel}.source_sha256_16") != source_sha(kernel):
        return None
    try:
        return float(vals[f"{kernel}.traffic_bytes"])
    except (KeyError, ValueError):
        return None


def roofline_entries(b, res):
    """Achieved vs peak for the two attention kernels, from the HIP-event
    medians of the timed multiplexed region; returns (dominant, other)."""
    n_launch = len(b.chunks)
    pre_ms = res["mux"]["prefill_kernel_ms"] / n_launch
    dec_ms = res["mux"]["decode_kernel_ms"]
    split = res["mux"]["prefill_kernels"] > 1   # key-range split: split + merge kernels per call
    pre = {"kernel": "k_prefill_split+k_prefill_merge" if split else "k_prefill_attn", "bound": "mfma",
           "unit": "TFLOP/s",
           "achieved": b.pre_flop / n_launch / (pre_ms * 1e-3) / 1e12, "peak": BF16_PEAK_TFLOPS,
           "work_per_launch": b.pre_flop / n_launch, "work_unit": "FLOP", "kernel_ms": pre_ms,
           "launches_per_step": n_launch}
    pre["frac"] = pre["achieved"] / pre["peak"]
    pre["share_peak"] = BF16_PEAK_TFLOPS * res["prefill_cus"] / N_CU
    pre["frac_share"] = pre["achieved"] / pre["share_peak"]
    pre["mfma_ceiling_tflops"] = res["prefill_mfma_ceiling_tflops"]
    pre["frac_ceiling"] = pre["achieved"] / pre["mfma_ceiling_tflops"]
    dec = {"kernel": "k_decode_balanced", "bound": "hbm", "unit": "GB/s",
           "achieved": b.dec_bytes / (dec_ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
           "work_per_launch": b.dec_bytes, "work_unit": "B", "kernel_ms": dec_ms,
           "launches_per_step": res["decode_iters_per_step"]}
    dec["frac"] = dec["achieved"] / dec["peak"]
    dec["measured_ceiling"] = res["decode_partition_stream_read_gbs"]
    dec["frac_measured"] = dec["achieved"] / dec["measured_ceiling"]
    dec["share_peak"] = HBM_PEAK_GBS * res["decode_cus"] / N_CU
    dec["frac_share"] = dec["achieved"] / dec["share_peak"]
    for e in (pre, dec):
        e["traffic"] = committed_traffic(e["kernel"], b.cfg.name)
    # dominant = the larger share of the step's GPU time
    dec_total = dec_ms * res["decode_iters_per_step"]
    return (pre, dec) if res["mux"]["prefill_kernel_ms"] >= dec_total else (dec, pre)


# -------------------------------------------------------- one partition --
def run_partition(b, p_cus, d_cus, p_index, args):
    torch = b.torch
    part = b.Partition(p_cus, d_cus)
    try:
        ps, ds = part.prefill_stream, part.decode_stream
        reps = args.iso_reps
        for _ in range(max(1, args.warmup)):
            b.prefill_call(ps)
            b.decode_call(ds)
        torch.cuda.synchronize()
        iso_p = b.isolated("prefill", ps, reps)
        iso_d = b.isolated("decode", ds, reps)
        solo_p = b.isolated("prefill", b.gpu.full.cuda_stream, reps)
        solo_d = b.isolated("decode", b.gpu.full.cuda_stream, reps)
        ceiling = b.gpu.stream_ceiling(ds, d_cus)
        mfma_ceiling = b.gpu.mfma_ceiling(ps, p_cus)
        # isolated outputs, for the bit-exact comparison with multiplexed ones
        b.prefill_call(ps)
        b.decode_call(ds)
        torch.cuda.synchronize()
        ref_pre, ref_dec = b.dw.o_pre.clone(), b.dw.o_dec.clone()
        tp = median(iso_p["call"])
        td = median(iso_d["call"])
        m = max(1, int(round(tp / td)))
        # warm-up of the multiplexed loop; the decode iterations per step are
        # then taken from its multiplexed times, so that the decode stream stays
        # busy for the whole prefill window (isolated times understate the
        # prefill's slowdown and would leave the last prefill launches alone)
        warm = b.multiplexed(part, max(2, args.warmup), m)
        m_mux = max(1, int(round(median(warm["prefill_k"]) / median(warm["decode_call"]))))
        log(f"[bench] {b.cfg.name} {p_cus}/{d_cus}: isolated prefill {tp:.3f} ms, decode {td:.3f} ms; "
            f"multiplexed {median(warm['prefill_k']):.3f} / {median(warm['decode_call']):.3f} ms "
            f"-> {m_mux} decode iteration(s) per step")
        if m_mux != m:
            m = m_mux
            b.multiplexed(part, max(1, args.warmup), m)
        b.dw.o_pre.zero_()
        b.dw.o_dec.zero_()
        mux = b.multiplexed(part, args.steps, m, MARK_BASE + 64 * b.index + 2 * p_index)
        same = bool(torch.equal(ref_pre, b.dw.o_pre) and torch.equal(ref_dec, b.dw.o_dec))
    finally:
        part.close()
    steps, wall = args.steps, mux["wall_s"]
    res = {
        "prefill_cus": p_cus, "decode_cus": d_cus, "decode_iters_per_step": m,
        "ms_per_step": 1e3 * wall / steps,
        "prefill_tflops": steps * b.pre_flop / wall / 1e12,
        "decode_gbs": steps * m * b.dec_bytes / wall / 1e9,
        "iso": {"prefill_kernel_ms": median(iso_p["k0"]), "decode_kernel_ms": median(iso_d["k0"]),
                "decode_kernels": iso_d["kernels"], "decode_call_ms": median(iso_d["call"]),
                "flushed": True},
        "solo_full_gpu": {"prefill_kernel_ms": median(solo_p["k0"]), "decode_call_ms": median(solo_d["call"])},
        "mux": {"prefill_kernel_ms": median(mux["prefill_k"]), "prefill_kernel_p90_ms": p90(mux["prefill_k"]),
                "prefill_kernels": mux["prefill_kernels"],
                "decode_kernel_ms": median(mux["decode_k0"]), "decode_call_ms": median(mux["decode_call"]),
                "decode_call_p90_ms": p90(mux["decode_call"]),
                "prefill_window_ms": mux["prefill_window_ms"], "decode_window_ms": mux["decode_window_ms"]},
        "mux_equals_isolated_bitwise": same,
        "decode_partition_stream_read_gbs": ceiling,
        "prefill_mfma_ceiling_tflops": mfma_ceiling,
    }
    res["slowdown"] = {"prefill": res["mux"]["prefill_kernel_ms"] / res["iso"]["prefill_kernel_ms"],
                       "decode": res["mux"]["decode_call_ms"] / res["iso"]["decode_call_ms"]}
    dom, other = roofline_entries(b, res)
    res["roofline"], res["roofline_other"] = dom, other
    return res


# ----------------------------------------------- parity and CPU baseline --
def parity_rows(n: int) -> list:
    """Rows of every 64-position query block at the edges of its 16-row
    groups (offsets 0, 15, 16, 31, 32, 47, 48, 63), and the chunk's last row."""
    offs = (0, 15, 16, 31, 32, 47, 48, 63)
    return sorted({q + o for q in range(0, n, 64) for o in offs if q + o < n} | {n - 1})


def cpu_model():
    info = {}
    try:
        for line in open("/proc/cpuinfo"):
            if ":" in line:
                k, v = (x.strip() for x in line.split(":", 1))
                if k in ("model name", "cpu family", "model", "stepping") and k not in info:
                    info[k] = v
    except OSError:
        pass
    name = info.get("model name") or platform.processor() or "unknown"
    return f"{name} (family {info.get('cpu family', '?')}, model {info.get('model', '?')}, " \
           f"stepping {info.get('stepping', '?')})"


def parity_and_cpu(b):
    """The oracle on the multiplexed outputs of the timed region: every decode
    sequence, each prefill chunk's block-edge rows (all rows of the tiny
    workload).  Per call max-abs / mean-abs over the compared elements; the
    oracle's own time on these rows is the workload's CPU baseline."""
    import oracle
    from paper_2504_14489_amd import accounting
    from paper_2504_14489_amd.device import to_bits, bits_to_f32
    wl, cfg = b.wl, b.cfg
    b.torch.cuda.synchronize()
    o_pre, o_dec = to_bits(b.dw.o_pre), to_bits(b.dw.o_dec)
    threads = oracle.default_threads()
    calls, flop, pre_s, n_rows = [], 0, 0.0, 0
    for r, n in cfg.pre_chunks:
        rows = list(range(n)) if cfg.name in PARITY_ONLY else parity_rows(n)
        nvis = np.asarray([r + i + 1 for i in rows], dtype=np.int32)
        t = time.perf_counter()
        ref = oracle.paged_attention(wl.q_pre[[r + i for i in rows]], wl.k_pool, wl.v_pool, wl.pre_bt,
                                     np.zeros(len(rows), np.int32), nvis, n_threads=threads)
        pre_s += time.perf_counter() - t
        flop += sum(4 * cfg.head_dim * cfg.hq * int(v) for v in nvis)
        n_rows += len(rows)
        e = np.abs(bits_to_f32(o_pre[[r + i for i in rows]]) - ref)
        calls.append({"call": f"prefill r={r} n={n}", "rows": len(rows), "max_abs": float(e.max()),
                      "mean_abs": float(e.mean()), "finite": bool(np.all(np.isfinite(e)))})
    B = len(wl.dec_lens)
    t = time.perf_counter()
    ref = oracle.decode(wl.q_dec, wl.k_pool, wl.v_pool, wl.dec_bt, wl.dec_lens, n_threads=threads)
    dec_s = time.perf_counter() - t
    e = np.abs(bits_to_f32(o_dec) - ref)
    calls.append({"call": "decode", "sequences": B, "max_abs": float(e.max()), "mean_abs": float(e.mean()),
                  "finite": bool(np.all(np.isfinite(e)))})
    ok = all(c["finite"] and c["max_abs"] <= 2e-2 and c["mean_abs"] <= 2e-3 for c in calls)
    parity = {"pass": ok, "tolerance": {"max_abs": 2e-2, "mean_abs": 2e-3}, "calls": calls,
              "max_abs": max(c["max_abs"] for c in calls),
              "sample": "every decode sequence; prefill rows at the 16-row-group edges of every query block "
                        "(all rows for tiny); tests/test_gpu_configs.py compares every row of every chunk "
                        "except the long-context one"}
    dbytes = accounting.decode_bytes(cfg.hq, cfg.hkv, cfg.head_dim, wl.dec_lens)
    cpu = {"value": flop / pre_s / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
           "sample": f"prefill: {n_rows} rows of {sum(n for _, n in cfg.pre_chunks)} (all {cfg.hq} heads, "
                     f"{flop / 1e9:.2f} GFLOP in {pre_s:.1f}s); decode: all {B} sequences "
                     f"({dbytes / 1e9:.3f} GB in {dec_s:.2f}s)",
           "decode_value": dbytes / dec_s / 1e9, "decode_unit": "GB/s",
           "host_cores": os.cpu_count(), "threads_used": threads, "cpu_model": cpu_model(),
           "precision": "fp64"}
    return parity, cpu


# ---------------------------------------------------------- one workload --
def measure(name, index, args, gpu):
    b = Bench(name, args, gpu, index)
    try:
        cfg = b.cfg
        splits = list(zip(cfg.prefill_cus, cfg.decode_cus))
        if args.partition >= 0:
            splits = [splits[min(args.partition, len(splits) - 1)]]
        parts = [run_partition(b, p, d, i, args) for i, (p, d) in enumerate(splits)]
        best = min(parts, key=lambda r: r["ms_per_step"])
        m = best["decode_iters_per_step"]
        tb = {k: b.temporal(k, args.steps, m) for k in ("serial", "free", "fused")}
        base = {k: v[0] for k, v in tb.items()}
        baselines = {"spatial_ms_per_step": best["ms_per_step"],
                     "spatial_split": [best["prefill_cus"], best["decode_cus"]],
                     "serial_ms_per_step": base["serial"], "free_streams_ms_per_step": base["free"],
                     "fused_ms_per_step": base["fused"],
                     "spatial_speedup": {k: base[k] / best["ms_per_step"] for k in base},
                     "decode_iteration_ms": {"spatial": best["mux"]["decode_call_ms"],
                                             **{k: v[1] for k, v in tb.items()}}}
        log(f"[bench] {name} equal-work step: spatial {best['ms_per_step']:.3f} ms, serial {base['serial']:.3f}, "
            f"free streams {base['free']:.3f}, fused {base['fused']:.3f}")
        parity = cpu = None
        if not args.no_cpu_baseline:
            t = time.time()
            parity, cpu = parity_and_cpu(b)
            log(f"[bench] {name} parity {'pass' if parity['pass'] else 'FAIL'} (max-abs {parity['max_abs']:.3g}), "
                f"oracle {cpu['value'] * 1e3:.1f} GFLOP/s, {cpu['decode_value']:.1f} GB/s, {time.time() - t:.1f}s")
        head = parts[0]
        return {"name": name, "workload": DESC[name], "parity_only": name in PARITY_ONLY,
                "prefill_chunks": [list(c) for c in cfg.pre_chunks], "decode_batch": int(len(b.wl.dec_lens)),
                "prefill_flop_per_step": b.pre_flop, "decode_bytes_per_iter": b.dec_bytes,
                "pool_replicas": b.replicas, "partitions": parts, "roofline": head["roofline"],
                "roofline_other": head["roofline_other"], "temporal_baselines": baselines,
                "parity": parity, "cpu_baseline": cpu}
    finally:
        b.close()
        b.torch.cuda.synchronize()
        b.torch.cuda.empty_cache()


# ----------------------------------------------------------- traffic pass --
def traffic_pass(args):
    """One isolated launch of each kernel on its partition, then a device copy
    of known size for the counter calibration."""
    import torch
    gpu = Device()
    b = Bench(args.names[0], args, gpu, 0)
    part = b.Partition(b.cfg.prefill_cus[0], b.cfg.decode_cus[0])
    try:
        b.prefill_call(part.prefill_stream)
        torch.cuda.synchronize()
        b.decode_call(part.decode_stream)
        torch.cuda.synchronize()
        src = torch.empty(256 << 20, dtype=torch.uint8, device=b.dw.device)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
    finally:
        part.close()
        b.close()
    log(f"[bench] traffic pass done: {b.cfg.name}, copy of {256 << 20} bytes")


def tables(entries):
    """Markdown: one row per workload (its first split), then the sweep."""
    rows = ["| workload | CUs pre/dec | prefill kernel (mux) | TFLOP/s | % share | % MFMA ceiling | decode kernel (mux) | "
            "GB/s | % stream ceiling | % of 8 TB/s | slowdown pre / dec | mux = iso | parity max-abs |",
            "|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for e in entries.values():
        r = e["partitions"][0]
        pre = r["roofline"] if r["roofline"]["bound"] == "mfma" else r["roofline_other"]
        dec = r["roofline_other"] if pre is r["roofline"] else r["roofline"]
        rows.append(f"| {e['name']} | {r['prefill_cus']}/{r['decode_cus']} | {pre['kernel_ms']:.3f} ms | "
                    f"{pre['achieved']:.1f} | {100 * pre['frac_share']:.1f} | {100 * pre['frac_ceiling']:.1f} | "
                    f"{dec['kernel_ms']:.3f} ms | {dec['achieved']:.0f} | {100 * dec['frac_measured']:.1f} | "
                    f"{100 * dec['frac']:.1f} | {r['slowdown']['prefill']:.3f} / {r['slowdown']['decode']:.3f} | "
                    f"{r['mux_equals_isolated_bitwise']} | "
                    f"{e['parity']['max_abs'] if e['parity'] else float('nan'):.2g} |")
    out = "\n".join(rows)
    sw = entries.get("sweep8b")
    if sw and len(sw["partitions"]) > 1:
        out += "\n\n" + sweep_table(sw)
    return out


def sweep_table(e):
    rows = ["| prefill CUs | prefill iso / mux ms | slowdown | TFLOP/s (mux) | % share | % MFMA ceiling | "
            "decode iso / mux ms | slowdown | GB/s (mux) | % stream ceiling | % share |",
            "|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in e["partitions"]:
        pre = r["roofline"] if r["roofline"]["bound"] == "mfma" else r["roofline_other"]
        dec = r["roofline_other"] if pre is r["roofline"] else r["roofline"]
        rows.append(f"| {r['prefill_cus']} | {r['iso']['prefill_kernel_ms']:.3f} / {r['mux']['prefill_kernel_ms']:.3f} | "
                    f"{r['slowdown']['prefill']:.3f} | {pre['achieved']:.1f} | {100 * pre['frac_share']:.1f} | "
                    f"{100 * pre['frac_ceiling']:.1f} | {r['iso']['decode_call_ms']:.3f} / "
                    f"{r['mux']['decode_call_ms']:.3f} | {r['slowdown']['decode']:.3f} | {dec['achieved']:.0f} | "
                    f"{100 * dec['frac_measured']:.1f} | {100 * dec['frac_share']:.1f} |")
    return "\n".join(rows)


def main():
    args = parse()
    if args.gpus != 1:
        log(f"bench.py runs on one GPU only: the multiplexed path partitions the compute units "
            f"of a single MI355X and has no multi-GPU mode (asked for --gpus {args.gpus}).")
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        log("bench.py needs a GPU")
        sys.exit(1)
    if args.traffic_pass:
        traffic_pass(args)
        return
    t_start = time.time()
    gpu = Device()
    entries = {}
    for name in args.names:
        entries[name] = measure(name, ORDER.index(name), args, gpu)
    h = entries[args.headline]
    head = h["partitions"][0]
    line = {
        "metric": METRIC,
        "value": round(head["prefill_tflops"], 3),
        "unit": "TFLOP/s",
        "decode_value": round(head["decode_gbs"], 1),
        "decode_unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(head["ms_per_step"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": h["workload"], "name": h["name"], "seed": args.seed,
                   "prefill_cus": head["prefill_cus"], "decode_cus": head["decode_cus"],
                   "decode_batch": h["decode_batch"], "prefill_chunks": h["prefill_chunks"],
                   "prefill_flop_per_step": h["prefill_flop_per_step"],
                   "decode_bytes_per_iter": h["decode_bytes_per_iter"],
                   "decode_iters_per_step": head["decode_iters_per_step"],
                   "pool_replicas": h["pool_replicas"]},
        "roofline": h["roofline"],
        "roofline_other": h["roofline_other"],
        "cpu_baseline": h["cpu_baseline"],
        "parity": h["parity"],
        "partitions": h["partitions"],
        "temporal_baselines": h["temporal_baselines"],
        "protocol": {"isolated_flushed_bytes": FLUSH_BYTES, "replicas_below_decode_kv_bytes": REPLICA_BELOW,
                     "iso_reps": args.iso_reps, "timed": "HIP events per kernel on its own stream; "
                     "value = prefill FLOP x steps / wall time of the timed region"},
        "configs": {k: v for k, v in entries.items() if k != args.headline},
        "bench_wall_s": round(time.time() - t_start, 1),
    }
    if "sweep8b" in entries and len(entries["sweep8b"]["partitions"]) > 1:
        line["contention_sweep"] = [
            {"prefill_cus": r["prefill_cus"], "decode_cus": r["decode_cus"],
             "prefill_iso_ms": r["iso"]["prefill_kernel_ms"], "prefill_mux_ms": r["mux"]["prefill_kernel_ms"],
             "prefill_slowdown": r["slowdown"]["prefill"], "decode_iso_ms": r["iso"]["decode_call_ms"],
             "decode_mux_ms": r["mux"]["decode_call_ms"], "decode_slowdown": r["slowdown"]["decode"]}
            for r in entries["sweep8b"]["partitions"]]
    print(json.dumps(line), flush=True)
    table = tables(entries)
    log(table)
    if args.table:
        with open(args.table, "w") as f:
            f.write(table + "\n")


if __name__ == "__main__":
    main()
