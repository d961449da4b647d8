"""Short text summaries of rocprofv3 output for the committed profiles.

    python -m paper_2504_14489_amd.rocprof_summary traffic --workload llama8b \\
        --fetch <dir of the FETCH_SIZE run> --write <dir of the WRITE_SIZE run> --out profiles/traffic_llama8b.txt
    python -m paper_2504_14489_amd.rocprof_summary trace --stats-dir <dir of a --kernel-trace --stats run> \\
        --title "..." --command "..." --out profiles/kernel_trace_llama8b.md
    python -m paper_2504_14489_amd.rocprof_summary mfma --dir <dir of the MFMA counter run> --workload llama8b \\
        --cus 64 --out profiles/mfma_llama8b.txt

The traffic summary scales each kernel's FETCH_SIZE / WRITE_SIZE (KiB per
dispatch) by what the same counter reads for the runtime's device copy of a
known size in the same run, and records the kernel sources' hash so that a
reader (bench.py) can tell when the figures no longer describe the kernel.
"""
from __future__ import annotations

import argparse
import csv
import glob
import os
import re
import statistics
import sys
from collections import defaultdict

COPY_KERNEL = "__amd_rocclr_copyBuffer"
COPY_BYTES = 256 << 20        # the copy bench.py --traffic-pass makes
N_XCD = 8                     # accelerator dies of an MI355X


def _rows(d: str, suffix: str):
    files = sorted(glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True))
    if not files:
        raise SystemExit(f"no *{suffix} under {d}")
    for f in files:
        with open(f, newline="") as fh:
            yield from csv.DictReader(fh)


def _short(name: str) -> str:
    """Kernel name without template arguments, parameters or namespaces."""
    name = name.replace("(anonymous namespace)::", "")
    name = re.sub(r"^void ", "", name.strip())
    name = re.sub(r"\(.*$", "", name)
    name = re.sub(r"<.*>", "", name)
    return name.split("::")[-1].strip()


def counter_per_dispatch(d: str, counter: str):
    """kernel -> list of the counter's value per dispatch (summed over the
    rows a dispatch has, e.g. one per XCD)."""
    per = defaultdict(float)
    names = {}
    for r in _rows(d, "counter_collection.csv"):
        if r.get("Counter_Name") != counter:
            continue
        key = r.get("Dispatch_Id") or r.get("Correlation_Id")
        per[key] += float(r["Counter_Value"])
        names[key] = _short(r["Kernel_Name"])
    out = defaultdict(list)
    for k, v in per.items():
        out[names[k]].append(v)
    return out


def traffic(args):
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    from bench import source_sha, KERNEL_SOURCES
    fetch = counter_per_dispatch(args.fetch, "FETCH_SIZE")
    write = counter_per_dispatch(args.write, "WRITE_SIZE")
    if COPY_KERNEL not in fetch or COPY_KERNEL not in write:
        raise SystemExit("the calibration copy is missing from the counter runs")
    kib = COPY_BYTES / 1024
    # the calibration copy is the largest copy of the run (the others upload
    # the workload's small arrays)
    f_copy, w_copy = max(fetch[COPY_KERNEL]), max(write[COPY_KERNEL])
    f_scale, w_scale = kib / f_copy, kib / w_copy
    lines = [f"# HBM traffic per launch: {args.workload} workload", "",
             "Commands (on the MI355X box, from /tmp with TMPDIR=/tmp; one counter per run):", "",
             f"    rocprofv3 --pmc FETCH_SIZE --output-format csv -d {args.fetch} -o run -- "
             f"python3 bench.py --config {args.workload} --traffic-pass",
             f"    rocprofv3 --pmc WRITE_SIZE --output-format csv -d {args.write} -o run -- "
             f"python3 bench.py --config {args.workload} --traffic-pass",
             f"    python -m paper_2504_14489_amd.rocprof_summary traffic --workload {args.workload} "
             f"--fetch {args.fetch} --write {args.write} --out <this file>", "",
             "bench.py --traffic-pass runs one isolated launch of each kernel on its partition and a "
             f"device-to-device copy of {COPY_BYTES} bytes ({COPY_KERNEL}) that calibrates the counters.", "",
             f"# copy calibration: FETCH_SIZE read {f_copy:.1f} KiB and WRITE_SIZE {w_copy:.1f} KiB for "
             f"{kib:.0f} KiB moved",
             f"copy.fetch_scale: {f_scale:.4f}", f"copy.write_scale: {w_scale:.4f}", ""]
    for k in sorted(set(fetch) & set(write)):
        if k == COPY_KERNEL or not k.startswith("k_"):
            continue
        fk, wk = statistics.median(fetch[k]), statistics.median(write[k])
        tb = (fk * f_scale + wk * w_scale) * 1024
        lines += [f"# {k}: FETCH_SIZE {fk:.1f} KiB, WRITE_SIZE {wk:.1f} KiB per dispatch (raw, median of "
                  f"{len(fetch[k])})", f"{k}.fetch_kib: {fk:.3f}", f"{k}.write_kib: {wk:.3f}",
                  f"{k}.traffic_bytes: {tb:.0f}"]
        if k in KERNEL_SOURCES:
            lines.append(f"{k}.source_sha256_16: {source_sha(k)}")
        lines.append("")
    with open(args.out, "w") as f:
        f.write("\n".join(lines))
    print("\n".join(lines))


def mfma(args):
    """Matrix-core use of k_prefill_attn from SQ_INSTS_VALU_MFMA_MOPS_BF16 (512 flop
    each), SQ_VALU_MFMA_BUSY_CYCLES (summed over SIMDs) and GRBM_GUI_ACTIVE."""
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    from bench import source_sha
    from paper_2504_14489_amd import accounting, workloads as W
    cfg = W.CONFIGS[args.workload]
    vals = {c: counter_per_dispatch(args.dir, c) for c in
            ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE")}
    k = "k_prefill_attn"
    mops = statistics.median(vals["SQ_INSTS_VALU_MFMA_MOPS_BF16"][k])
    busy = statistics.median(vals["SQ_VALU_MFMA_BUSY_CYCLES"][k])
    # the CSV sums GRBM_GUI_ACTIVE over the 8 XCDs; each XCD counts the same
    # dispatch, so one XCD's count is the dispatch's duration in cycles
    active = statistics.median(vals["GRBM_GUI_ACTIVE"][k]) / N_XCD
    algo = accounting.prefill_flops(cfg.hq, cfg.head_dim, [cfg.pre_chunks[0]])
    simds = 4 * args.cus
    lines = [f"# Matrix-core use of k_prefill_attn: {args.workload} workload, first prefill chunk on {args.cus} CUs",
             "", "Commands (on the MI355X box, from /tmp with TMPDIR=/tmp):", "",
             f"    rocprofv3 --pmc SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE "
             f"--output-format csv -d {args.dir} -o run -- python3 bench.py --config {args.workload} "
             f"--traffic-pass",
             f"    python -m paper_2504_14489_amd.rocprof_summary mfma --dir {args.dir} --workload "
             f"{args.workload} --cus {args.cus} --out <this file>", "",
             f"k_prefill_attn.mfma_bf16_flop: {mops * 512:.0f}",
             f"k_prefill_attn.algorithmic_flop: {algo:.0f}",
             f"k_prefill_attn.executed_over_algorithmic: {mops * 512 / algo:.4f}",
             f"k_prefill_attn.mfma_busy_cycles_sum: {busy:.0f}",
             f"k_prefill_attn.gui_active_cycles_per_xcd: {active:.0f}",
             f"k_prefill_attn.mfma_busy_fraction_of_partition_simds: {busy / (active * simds):.4f}",
             f"k_prefill_attn.source_sha256_16: {source_sha(k)}", "",
             "executed / algorithmic > 1: the MFMAs of masked key tiles on the diagonal and of padding rows.",
             "busy fraction: SQ_VALU_MFMA_BUSY_CYCLES over GRBM_GUI_ACTIVE times the partition's SIMDs "
             f"({simds}).", ""]
    with open(args.out, "w") as f:
        f.write("\n".join(lines))
    print("\n".join(lines))


def trace(args):
    rows = list(_rows(args.stats_dir, "kernel_stats.csv"))
    tot = sum(float(r["TotalDurationNs"]) for r in rows)
    lines = [f"# {args.title}", "", "Command (on the MI355X box, from /tmp with TMPDIR=/tmp):", "",
             f"    {args.command}", "", "## --stats summary (all dispatches of the run)", "",
             "| kernel | calls | average (us) | min (us) | max (us) | share of GPU time |",
             "|---|---|---|---|---|---|"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        lines.append(f"| {_short(r['Name'])[:40]} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                     f"{100 * float(r['TotalDurationNs']) / tot:.1f}% |")
    if args.trace_last:
        # per-dispatch durations of the last N dispatches of each kernel
        disp = defaultdict(list)
        for r in _rows(args.stats_dir, "kernel_trace.csv"):
            disp[_short(r["Kernel_Name"])].append(
                (int(r["Start_Timestamp"]), int(r["End_Timestamp"]) - int(r["Start_Timestamp"])))
        skip = f" before the last {args.skip_last}" if args.skip_last else ""
        lines += ["", f"## The last {args.trace_last} dispatches{skip} of each kernel (the timed region)", "",
                  "| kernel | mean (us) | median (us) |", "|---|---|---|"]
        for k in args.kernels.split(","):
            if k in disp:
                seq = [d for _, d in sorted(disp[k])]
                seq = seq[:len(seq) - args.skip_last] if args.skip_last else seq
                last = seq[-args.trace_last:]
                lines.append(f"| {k} | {statistics.mean(last) / 1e3:.1f} | {statistics.median(last) / 1e3:.1f} |")
    if args.regions:
        lines += marked_regions(args.stats_dir, args.kernels.split(","))
    if args.note:
        lines += ["", args.note]
    with open(args.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def marked_regions(d: str, kernels):
    """Per-kernel durations inside each timed region the benchmark marked:
    k_trace_mark dispatches of id MARK_BASE + 64 w + 2 p open the region of
    workload w (bench.ORDER), CU split p on both streams and id + 1 closes it;
    a kernel belongs to the region when its dispatch starts inside it."""
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    from bench import MARK_BASE, ORDER
    marks = defaultdict(list)
    disp = []
    for r in _rows(d, "kernel_trace.csv"):
        name = _short(r["Kernel_Name"])
        t0, t1 = int(r["Start_Timestamp"]), int(r["End_Timestamp"])
        if name == "k_trace_mark":
            marks[int(r["Grid_Size_X"]) // int(r["Workgroup_Size_X"])].append((t0, t1))
        elif name in kernels:
            disp.append((t0, t1, name))
    out = ["", "## Timed regions marked by bench.py (dispatches starting between the marks)", "",
           "| workload | split | kernel | dispatches | mean (us) | median (us) |", "|---|---|---|---|---|---|"]
    for mid in sorted(marks):
        if (mid - MARK_BASE) % 2 or mid + 1 not in marks:
            continue
        lo, hi = min(t for t, _ in marks[mid]), max(t for _, t in marks[mid + 1])
        w, p = divmod(mid - MARK_BASE, 64)
        for k in kernels:
            ds = [(t1 - t0) / 1e3 for t0, t1, n in disp if n == k and lo <= t0 <= hi]
            if ds:
                out.append(f"| {ORDER[w] if w < len(ORDER) else w} | {p // 2} | {k} | {len(ds)} | "
                           f"{statistics.mean(ds):.1f} | {statistics.median(ds):.1f} |")
    return out


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    t = sub.add_parser("traffic")
    t.add_argument("--workload", required=True)
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--out", required=True)
    k = sub.add_parser("trace")
    k.add_argument("--stats-dir", required=True)
    k.add_argument("--title", required=True)
    k.add_argument("--command", required=True)
    k.add_argument("--trace-last", type=int, default=0)
    k.add_argument("--skip-last", type=int, default=0)
    k.add_argument("--kernels", default="k_prefill_attn,k_decode_balanced")
    k.add_argument("--note", default="")
    k.add_argument("--regions", action="store_true", help="durations inside the regions bench.py marked")
    k.add_argument("--out", required=True)
    m = sub.add_parser("mfma")
    m.add_argument("--dir", required=True)
    m.add_argument("--workload", required=True)
    m.add_argument("--cus", type=int, required=True)
    m.add_argument("--out", required=True)
    args = ap.parse_args(argv)
    {"traffic": traffic, "trace": trace, "mfma": mfma}[args.cmd](args)


if __name__ == "__main__":
    main()
