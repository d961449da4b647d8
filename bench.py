#!/usr/bin/env python3
"""Benchmark: paged GQA prefill + decode attention multiplexed on split CUs.

One step = one pass of the whole hot path over one batch of synthetic input,
with the two phases on disjoint CU partitions of the GPU (decode enqueued
first, as the paper launches the decode iteration before prefill, Sec. 3.2.2):

  decode stream : m x (append each sequence's new K/V, decode attention
                  = split kernel + combine kernel)
  prefill stream: append the chunk's new K/V, causal prefill attention

m is the number of decode iterations that fit in one prefill call on the
isolated partitions (at least 1), so both partitions stay busy for the whole
timed region, as in the paper's bubble-less multiplexing.

Printed (one JSON line on stdout): prefill TFLOP/s and decode HBM GB/s over
the timed region, isolated and multiplexed per-call latencies, the contention
slowdown, the roofline of the dominant kernel, and the CPU oracle's rate on a
bounded sample of the same workload.  Progress goes to stderr.
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


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="llama8b",
                    help="tiny | llama8b | llama70b | longctx8b | sweep8b")
    ap.add_argument("--partition", type=int, default=-1,
                    help="index into the config's CU splits (sweep8b has 7); -1 = all")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--iso-reps", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle baseline sample")
    ap.add_argument("--no-parity", action="store_true")
    ap.add_argument("--table", default="", help="also write the per-partition table (Markdown) here")
    ap.add_argument("--traffic-pass", action="store_true",
                    help="run each kernel once on its partition plus a device copy of known size "
                         "(the command profiled by rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE), then exit")
    return ap.parse_args()


def median(x):
    return statistics.median(x) if x else float("nan")


def p90(x):
    return float(np.percentile(x, 90)) if x else float("nan")


class Bench:
    def __init__(self, args):
        import torch
        from paper_2504_14489_amd import accounting, workloads as W
        from paper_2504_14489_amd.device import DeviceWorkload, Partition, Timing, _dev16

        self.torch = torch
        self.Timing = Timing
        self.Partition = Partition
        self.args = args
        self.cfg = W.CONFIGS[args.config]
        t = time.time()
        self.wl = W.make_workload(self.cfg, seed=args.seed)
        log(f"[bench] workload {self.cfg.name}: {self.wl.num_pages} pages, "
            f"{len(self.wl.dec_lens)} decodes, generated in {time.time() - t:.1f}s")
        self.dw = DeviceWorkload(self.wl)
        c = self.cfg
        self.chunks = list(c.pre_chunks)
        self.pre_flop = accounting.prefill_flops(c.hq, c.head_dim, self.chunks)
        self.dec_bytes = accounting.decode_bytes(c.hq, c.hkv, c.head_dim, self.wl.dec_lens)
        # the step's appended K/V rows (bit-identical to what the pool holds)
        self.pre_new = [tuple(_dev16(a, self.dw.device) for a in self.wl.pre_new_kv(r, n))
                        for r, n in self.chunks]
        kd, vd = self.wl.dec_new_kv()
        self.dec_new = (_dev16(kd, self.dw.device), _dev16(vd, self.dw.device))
        self.full = torch.cuda.Stream()           # no CU mask: the whole GPU
        torch.cuda.synchronize()

    # ------------------------------------------------------------ phases --
    def prefill_call(self, stream, tw=None, tp=None):
        """All prefill chunks of the step: append, then attention."""
        for (r, n), (k, v) in zip(self.chunks, self.pre_new):
            self.dw.write_prefill_kv(r, n, k, v, stream, tw.h if tw else None)
            self.dw.prefill(r, n, stream, tp.h if tp else None)

    def decode_call(self, stream, tw=None, td=None):
        self.dw.write_decode_kv(self.dec_new[0], self.dec_new[1], stream, tw.h if tw else None)
        self.dw.decode(stream, td.h if td else None)

    # ---------------------------------------------------------- isolated --
    def isolated(self, which, stream, reps):
        """Per-call latency of one phase alone on `stream`: kernel ms lists."""
        torch = self.torch
        outs = {"call": [], "k0": [], "k1": [], "append": []}
        nchunk = len(self.chunks) if which == "prefill" else 1
        tws = [[self.Timing() for _ in range(nchunk)] for _ in range(reps)]
        tks = [[self.Timing() for _ in range(nchunk)] for _ in range(reps)]
        torch.cuda.synchronize()
        for i in range(reps):
            if which == "prefill":
                for (r, n), (k, v), tw, tk in zip(self.chunks, self.pre_new, tws[i], tks[i]):
                    self.dw.write_prefill_kv(r, n, k, v, stream, tw.h)
                    self.dw.prefill(r, n, stream, tk.h)
            else:
                self.decode_call(stream, tws[i][0], tks[i][0])
        torch.cuda.synchronize()
        for i in range(reps):
            outs["k0"].append(sum(tk.kernel_ms(0) for tk in tks[i]))
            outs["call"].append(sum(tk.elapsed()[0] for tk in tks[i]))
            if which == "decode":
                outs["k1"].append(tks[i][0].kernel_ms(1))
            outs["append"].append(sum(tw.elapsed()[0] for tw in tws[i]))
        return outs

    def stream_ceiling(self, stream, n_cus, nbytes=1 << 30, reps=5):
        """HBM read rate the CUs of `stream` reach on a plain 1 GiB stream."""
        from paper_2504_14489_amd import mw
        torch = self.torch
        if not hasattr(self, "_stream_buf"):
            self._stream_buf = torch.empty(nbytes, dtype=torch.uint8, device=self.dw.device)
            self._sink = torch.empty(1 << 16, dtype=torch.int32, device=self.dw.device)
        blocks = 8 * n_cus
        ts = [self.Timing() for _ in range(reps + 1)]
        torch.cuda.synchronize()
        for t in ts:
            mw.mw_stream_read(self._stream_buf.data_ptr(), nbytes, self._sink.data_ptr(), blocks,
                              stream, t.h)
        torch.cuda.synchronize()
        ms = median([t.kernel_ms(0) for t in ts[1:]])
        return nbytes / (ms * 1e-3) / 1e9

    # ------------------------------------------------------- multiplexed --
    def multiplexed(self, part, steps, m):
        torch = self.torch
        ps, ds = part.prefill_stream, part.decode_stream
        tp = [[self.Timing() for _ in self.chunks] for _ in range(steps)]
        td = [[self.Timing() for _ in range(m)] for _ in range(steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(steps):
            for j in range(m):                      # decode first
                self.decode_call(ds, None, td[k][j])
            for (r, n), (kk, vv), t in zip(self.chunks, self.pre_new, tp[k]):
                self.dw.write_prefill_kv(r, n, kk, vv, ps)
                self.dw.prefill(r, n, ps, t.h)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        pre_k = [sum(t.kernel_ms(0) for t in tp[k]) for k in range(steps)]
        dec_k0 = [t.kernel_ms(0) for k in range(steps) for t in td[k]]
        dec_call = [t.elapsed()[0] for k in range(steps) for t in td[k]]
        # windows of the two streams relative to the first decode call's start
        from paper_2504_14489_amd import mw
        ref = td[0][0].h
        p_start = min(mw.mw_timing_offsets(tp[k][0].h, ref)[0] for k in range(steps))
        p_stop = max(mw.mw_timing_offsets(tp[k][-1].h, ref)[1] for k in range(steps))
        d_stop = mw.mw_timing_offsets(td[-1][-1].h, ref)[1]
        return {"wall_s": wall, "prefill_k": pre_k, "decode_k0": dec_k0, "decode_call": dec_call,
                "prefill_window_ms": [p_start, p_stop], "decode_window_ms": [0.0, d_stop]}

    # --------------------------------------------- temporal baselines --
    def temporal(self, kind, steps, m):
        """Wall ms per step of the same work without CU partitions, on the
        whole GPU: "serial" = prefill, then m decode iterations, one stream;
        "free" = the two phases on two unmasked streams (the hardware shares
        the CUs); "fused" = appends, one fused prefill + decode launch, then
        m - 1 more decode iterations."""
        torch = self.torch
        from paper_2504_14489_amd import mw
        s1 = self.full.cuda_stream
        if not hasattr(self, "full2"):
            self.full2 = torch.cuda.Stream()
            self.eng_dec, self.eng_pre = self.dw.engine_args()

        td = []

        def step(timed=False):
            if kind == "serial":
                self.prefill_call(s1)
                for _ in range(m):
                    self.decode_call(s1)
            elif kind == "free":
                s2 = self.full2.cuda_stream
                for _ in range(m):
                    t = self.Timing() if timed else None
                    self.decode_call(s2, None, t)
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
    if not os.path.exists(path):
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


def traffic_pass(args):
    """One isolated launch of each kernel on its partition, then a device copy
    of known size for the counter calibration."""
    import torch
    b = Bench(args)
    p_cus, d_cus = b.cfg.prefill_cus[0], b.cfg.decode_cus[0]
    part = b.Partition(p_cus, d_cus)
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


def cpu_baseline(wl, cfg, seconds):
    """The oracle, as it stands, on a bounded sample of the same workload."""
    import oracle
    from paper_2504_14489_amd import accounting
    threads = max(1, min(16, os.cpu_count() or 1))
    r, n = cfg.pre_chunks[-1]
    # prefill rows spread evenly over the chunk (all heads); calibrate, then size
    def run_pre(k):
        idx = np.unique(np.linspace(0, n - 1, k).astype(int))
        t = time.perf_counter()
        for i in idx:
            oracle.prefill(wl.q_pre[r + i:r + i + 1], wl.k_pool, wl.v_pool, wl.pre_bt, r + i,
                           n_threads=threads)
        dt = time.perf_counter() - t
        flop = sum(4 * cfg.head_dim * cfg.hq * (r + i + 1) for i in idx)
        return dt, flop, len(idx)
    dt, flop, k = run_pre(4)
    k2 = int(min(n, max(4, 4 * (0.6 * seconds) / max(dt, 1e-3))))
    dt, flop, k = run_pre(k2)
    # decode: whole sequences (all heads), calibrated the same way
    B = len(wl.dec_lens)
    def run_dec(k):
        idx = np.unique(np.linspace(0, B - 1, k).astype(int))
        t = time.perf_counter()
        oracle.decode(wl.q_dec[idx], wl.k_pool, wl.v_pool, wl.dec_bt[idx], wl.dec_lens[idx],
                      n_threads=threads)
        return time.perf_counter() - t, accounting.decode_bytes(cfg.hq, cfg.hkv, cfg.head_dim,
                                                                wl.dec_lens[idx]), len(idx)
    ddt, dbytes, dk = run_dec(2)
    dk2 = int(min(B, max(2, 2 * (0.4 * seconds) / max(ddt, 1e-3))))
    ddt, dbytes, dk = run_dec(dk2)
    cpu = platform.processor() or ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": flop / dt / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"prefill: {k} of {n} rows of the last chunk (all {cfg.hq} heads, "
                      f"{flop / 1e9:.2f} GFLOP in {dt:.1f}s); decode: {dk} of {B} sequences "
                      f"({dbytes / 1e9:.3f} GB in {ddt:.1f}s)",
            "decode_value": dbytes / ddt / 1e9, "decode_unit": "GB/s", "cpu_model": cpu,
            "precision": "fp64"}


def parity(b, n_rows=24, n_seqs=8):
    """Sampled rows of the multiplexed outputs against the oracle."""
    import oracle
    from paper_2504_14489_amd.device import to_bits, bits_to_f32
    wl, cfg = b.wl, b.cfg
    torch = b.torch
    torch.cuda.synchronize()
    o_pre = to_bits(b.dw.o_pre)
    o_dec = to_bits(b.dw.o_dec)
    errs = []
    for r, n in cfg.pre_chunks:
        idx = np.unique(np.concatenate([[0, n - 1], np.linspace(0, n - 1, n_rows).astype(int)]))
        for i in idx:
            ref = oracle.prefill(wl.q_pre[r + i:r + i + 1], wl.k_pool, wl.v_pool, wl.pre_bt, r + i)
            errs.append(np.abs(bits_to_f32(o_pre[r + i:r + i + 1]) - ref))
    B = len(wl.dec_lens)
    sel = np.unique(np.linspace(0, B - 1, n_seqs).astype(int))
    ref = oracle.decode(wl.q_dec[sel], wl.k_pool, wl.v_pool, wl.dec_bt[sel], wl.dec_lens[sel])
    errs.append(np.abs(bits_to_f32(o_dec[sel]) - ref))
    e = np.concatenate([x.ravel() for x in errs])
    finite = bool(np.all(np.isfinite(bits_to_f32(o_pre))) and np.all(np.isfinite(bits_to_f32(o_dec))))
    return {"max_abs": float(e.max()), "mean_abs": float(e.mean()), "all_finite": finite,
            "rows_checked": int(sum(x.shape[0] for x in errs[:-1])), "seqs_checked": int(len(sel)),
            "pass": bool(finite and e.max() <= 2e-2 and e.mean() <= 2e-3)}


def run_partition(b, p_cus, d_cus, args):
    torch = b.torch
    part = b.Partition(p_cus, d_cus)
    try:
        ps, ds = part.prefill_stream, part.decode_stream
        reps = args.iso_reps
        # warm up both phases on their partitions
        for _ in range(max(1, args.warmup)):
            b.prefill_call(ps)
            b.decode_call(ds)
        torch.cuda.synchronize()
        iso_p = b.isolated("prefill", ps, reps)
        iso_d = b.isolated("decode", ds, reps)
        solo_p = b.isolated("prefill", b.full.cuda_stream, reps)
        solo_d = b.isolated("decode", b.full.cuda_stream, reps)
        ceiling = b.stream_ceiling(ds, d_cus)
        # isolated outputs, for the bit-exact comparison with multiplexed ones
        b.prefill_call(ps)
        b.decode_call(ds)
        torch.cuda.synchronize()
        ref_pre, ref_dec = b.dw.o_pre.clone(), b.dw.o_dec.clone()
        tp = median(iso_p["call"]) + median(iso_p["append"])
        td = median(iso_d["call"]) + median(iso_d["append"])
        m = max(1, int(round(tp / td)))
        log(f"[bench] partition {p_cus}/{d_cus}: isolated prefill {tp:.3f} ms, decode {td:.3f} ms "
            f"-> {m} decode iteration(s) per prefill call")
        b.multiplexed(part, max(1, args.warmup), m)    # warm-up of the multiplexed loop
        mux = b.multiplexed(part, args.steps, m)
        same = bool(torch.equal(ref_pre, b.dw.o_pre) and torch.equal(ref_dec, b.dw.o_dec))
    finally:
        part.close()
    steps = args.steps
    wall = mux["wall_s"]
    res = {
        "prefill_cus": p_cus, "decode_cus": d_cus, "decode_iters_per_step": m,
        "ms_per_step": 1e3 * wall / steps,
        "prefill_tflops": steps * b.pre_flop / wall / 1e12,
        "decode_gbs": steps * m * b.dec_bytes / wall / 1e9,
        "iso": {
            "prefill_kernel_ms": median(iso_p["k0"]), "prefill_append_ms": median(iso_p["append"]),
            "decode_split_ms": median(iso_d["k0"]), "decode_combine_ms": median(iso_d["k1"]),
            "decode_call_ms": median(iso_d["call"]), "decode_append_ms": median(iso_d["append"]),
        },
        "solo_full_gpu": {"prefill_kernel_ms": median(solo_p["k0"]), "decode_call_ms": median(solo_d["call"])},
        "mux": {
            "prefill_kernel_ms": median(mux["prefill_k"]), "prefill_kernel_p90_ms": p90(mux["prefill_k"]),
            "decode_split_ms": median(mux["decode_k0"]), "decode_call_ms": median(mux["decode_call"]),
            "decode_call_p90_ms": p90(mux["decode_call"]),
            "prefill_window_ms": mux["prefill_window_ms"], "decode_window_ms": mux["decode_window_ms"],
        },
        "mux_equals_isolated_bitwise": same,
        "decode_partition_stream_read_gbs": ceiling,
    }
    res["slowdown"] = {
        "prefill": res["mux"]["prefill_kernel_ms"] / res["iso"]["prefill_kernel_ms"],
        "decode": res["mux"]["decode_call_ms"] / res["iso"]["decode_call_ms"],
    }
    return res


def roofline_entries(b, res):
    """Achieved vs peak for the two dominant kernels, from event-timed means."""
    pre_ms = res["mux"]["prefill_kernel_ms"]
    dec_ms = res["mux"]["decode_split_ms"]
    pre_flop_launch = b.pre_flop / len(b.chunks)
    pre_ms_launch = pre_ms / len(b.chunks)
    pre = {"kernel": "k_prefill_attn", "bound": "mfma", "unit": "TFLOP/s",
           "achieved": pre_flop_launch / (pre_ms_launch * 1e-3) / 1e12, "peak": BF16_PEAK_TFLOPS,
           "work_per_launch": pre_flop_launch, "kernel_ms": pre_ms_launch}
    pre["frac"] = pre["achieved"] / pre["peak"]
    pre["share_peak"] = BF16_PEAK_TFLOPS * res["prefill_cus"] / N_CU
    pre["frac_share"] = pre["achieved"] / pre["share_peak"]
    dec = {"kernel": "k_decode_balanced", "bound": "hbm", "unit": "GB/s",
           "achieved": b.dec_bytes / (dec_ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
           "work_per_launch": b.dec_bytes, "kernel_ms": dec_ms}
    dec["frac"] = dec["achieved"] / dec["peak"]
    dec["share_peak"] = HBM_PEAK_GBS * res["decode_cus"] / N_CU
    dec["frac_share"] = dec["achieved"] / dec["share_peak"]
    dec["measured_ceiling"] = res["decode_partition_stream_read_gbs"]
    dec["frac_measured"] = dec["achieved"] / dec["measured_ceiling"]
    for e in (pre, dec):
        e["traffic"] = committed_traffic(e["kernel"], b.cfg.name)
    # dominant = larger share of the step's GPU time
    pre_total = pre_ms
    dec_total = dec_ms * res["decode_iters_per_step"]
    return (pre, dec) if pre_total >= dec_total else (dec, pre)


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
    b = Bench(args)
    cfg = b.cfg
    splits = list(zip(cfg.prefill_cus, cfg.decode_cus))
    if args.partition >= 0:
        splits = [splits[args.partition]]
    results = []
    for p_cus, d_cus in splits:
        results.append(run_partition(b, p_cus, d_cus, args))
    par = None if args.no_parity else parity(b)
    # the paper's core comparison (spatial vs temporal or fused sharing) at
    # equal work: the same step on the whole GPU without partitions
    m = results[0]["decode_iters_per_step"]
    res = {k: b.temporal(k, args.steps, m) for k in ("serial", "free", "fused")}
    base = {k: v[0] for k, v in res.items()}
    spatial = results[0]["ms_per_step"]
    spatial_dec = results[0]["mux"]["decode_call_ms"]
    best = min((r for r in results if r["decode_iters_per_step"] == m), key=lambda r: r["ms_per_step"])
    baselines = {"spatial_ms_per_step": spatial, "serial_ms_per_step": base["serial"],
                 "spatial_best_ms_per_step": best["ms_per_step"],
                 "spatial_best_split": [best["prefill_cus"], best["decode_cus"]],
                 "free_streams_ms_per_step": base["free"], "fused_ms_per_step": base["fused"],
                 "spatial_speedup": {k: base[k] / spatial for k in base},
                 "decode_iteration_ms": {"spatial": spatial_dec, **{k: v[1] for k, v in res.items()}}}
    log(f"[bench] equal-work step: spatial {spatial:.3f} ms, serial {base['serial']:.3f}, "
        f"free streams {base['free']:.3f}, fused {base['fused']:.3f}; decode iteration: spatial "
        f"{spatial_dec:.3f}, serial {res['serial'][1]:.3f}, free {res['free'][1]:.3f}, fused {res['fused'][1]:.3f}")
    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample ...")
        cpu = cpu_baseline(b.wl, cfg, args.cpu_seconds)
    b.close()

    head = results[0]
    dom, other = roofline_entries(b, head)
    desc = {
        "tiny": "tiny layer: 8 q-heads/2 kv-heads, 256-token prefill, 4 decodes U[128,512]",
        "llama8b": "Llama-3-8B-shaped attention layer: 32 q-heads/8 kv-heads, d=128, 16-token pages; "
                   "2048-token prefill chunk (no prefix) + 64 decodes with contexts U[512,4096]",
        "llama70b": "Llama-3-70B-shaped attention layer: 64 q-heads/8 kv-heads; 8192-token prefill in "
                    "four 2048-token chunks + 128 decodes, lognormal contexts (median 2048, sigma 0.8)",
        "llama70b_tp8": "one GPU's tensor-parallel-8 shard of the Llama-3-70B attention layer: 8 q-heads/1 kv-head; "
                        "8192-token prefill in four 2048-token chunks + 128 decodes, lognormal contexts",
        "longctx8b": "8B shapes, long context: 4096 new tokens over a 28672-token prefix + 32 decodes "
                     "U[16384,32768]",
        "sweep8b": "8B shapes: 4096-token prefill + 256 decodes U[1024,8192], prefill CU sweep",
    }[cfg.name]
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
        "config": {"workload": desc, "name": cfg.name, "seed": args.seed,
                   "prefill_cus": head["prefill_cus"], "decode_cus": head["decode_cus"],
                   "decode_batch": int(len(b.wl.dec_lens)),
                   "prefill_chunks": [list(c) for c in cfg.pre_chunks],
                   "prefill_flop_per_step": b.pre_flop,
                   "decode_bytes_per_iter": b.dec_bytes,
                   "decode_iters_per_step": head["decode_iters_per_step"]},
        "roofline": dom,
        "roofline_other": other,
        "cpu_baseline": cpu,
        "partitions": results,
        "temporal_baselines": baselines,
        "parity": par,
    }
    print(json.dumps(line), flush=True)
    if args.table or len(results) > 1:
        rows = ["| prefill CUs | prefill iso / mux ms | slowdown | TFLOP/s (mux) | % of share peak | "
                "decode iso / mux ms | slowdown | GB/s (mux) | % of share peak |",
                "|---|---|---|---|---|---|---|---|---|"]
        for r in results:
            pk = r["mux"]["prefill_kernel_ms"] / len(b.chunks)
            tf = b.pre_flop / len(b.chunks) / (pk * 1e-3) / 1e12
            gb = b.dec_bytes / (r["mux"]["decode_split_ms"] * 1e-3) / 1e9
            rows.append(
                f"| {r['prefill_cus']} | {r['iso']['prefill_kernel_ms']:.3f} / {r['mux']['prefill_kernel_ms']:.3f} | "
                f"{r['slowdown']['prefill']:.3f} | {tf:.1f} | {100 * tf / (BF16_PEAK_TFLOPS * r['prefill_cus'] / N_CU):.1f} | "
                f"{r['iso']['decode_call_ms']:.3f} / {r['mux']['decode_call_ms']:.3f} | {r['slowdown']['decode']:.3f} | "
                f"{gb:.0f} | {100 * gb / (HBM_PEAK_GBS * r['decode_cus'] / N_CU):.1f} |")
        table = "\n".join(rows)
        log(table)
        if args.table:
            with open(args.table, "w") as f:
                f.write(table + "\n")


if __name__ == "__main__":
    main()
