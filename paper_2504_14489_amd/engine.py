"""The bubble-less multiplex engine (paper Sec. 3.2) driven from Python, and
its measurement.

:class:`Engine` owns an ``mw_engine`` (a group of CU partitions created once)
and runs a plan through ``mw_engine_run``; every launch and every poll happens
in the library's host loop.  ``main`` measures, on one workload, what the
paper reports for its engine: the cost of creating the partition group and
its device memory, the repartition (switch) cost, the bubble ratio of the
two compute streams under blocking and polled coordination, and the overhead
of launching prefill layer by layer.

    python -m paper_2504_14489_amd.engine --config llama8b --out engine.json
"""
from __future__ import annotations

import argparse
import json
import statistics
import sys
from typing import Dict, List, Sequence

import numpy as np

from . import mw


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class Engine:
    def __init__(self, prefill_cus: Sequence[int], device: int = 0):
        self.h = mw.mw_engine_create(device, list(prefill_cus))
        self.prefill_cus = list(prefill_cus)

    def streams(self, config: int):
        """(prefill, decode) stream handles of partition `config` (-1: the whole device)."""
        return mw.mw_engine_streams(self.h, config)

    def memory(self):
        """(device bytes taken by creating the group, creation time in ms)."""
        return mw.mw_engine_memory(self.h)

    def run(self, dec: dict, pre: dict, *, config: int = 0, decode_iters: int, decode_layers: int,
            prefill_layers: int, layers_per_launch: int, policy: int = mw.MW_ENGINE_POLLED,
            switch_on_decode_end: bool = True, decode_graph: bool = False) -> dict:
        plan = mw.EnginePlan(config, decode_iters, decode_layers, prefill_layers, layers_per_launch,
                             policy, int(switch_on_decode_end), int(decode_graph))
        return mw.mw_engine_run(self.h, dec, pre, plan)

    def graphs(self):
        """(captured decode graphs, their device bytes, capture ms)."""
        return mw.mw_engine_graphs(self.h)

    def timeline(self, phase: int):
        return mw.mw_engine_timeline(self.h, phase)

    def close(self):
        if self.h is not None:
            mw.mw_engine_destroy(self.h)
            self.h = None


def _median_stats(runs: List[dict]) -> dict:
    return {k: statistics.median(r[k] for r in runs) for k in runs[0]}


def gap_stats(tl, decode_layers: int) -> dict:
    """Idle gaps on the decode stream from a timeline: between iterations
    (host-paced) and between calls inside one (queued back to back)."""
    gaps = tl[1:, 0] - tl[:-1, 1]
    at_boundary = (np.arange(1, len(tl)) % decode_layers) == 0
    g_it, g_call = gaps[at_boundary], gaps[~at_boundary]
    med = lambda g: float(np.median(g)) if len(g) else 0.0
    return {"iter_gap_ms_median": med(g_it), "iter_gap_ms_max": float(g_it.max()) if len(g_it) else 0.0,
            "call_gap_ms_median": med(g_call)}


# Coordination variants: (N_PL from the formula, total prefill layers) -> plan fields
VARIANTS = {
    "blocking": lambda n_pl, p: dict(policy=mw.MW_ENGINE_BLOCKING, layers_per_launch=p, switch_on_decode_end=False),
    "polled": lambda n_pl, p: dict(policy=mw.MW_ENGINE_POLLED, layers_per_launch=n_pl, switch_on_decode_end=False),
    "polled_switch": lambda n_pl, p: dict(policy=mw.MW_ENGINE_POLLED, layers_per_launch=n_pl,
                                          switch_on_decode_end=True),
    "polled_layer1": lambda n_pl, p: dict(policy=mw.MW_ENGINE_POLLED, layers_per_launch=1,
                                          switch_on_decode_end=False),
    "polled_all": lambda n_pl, p: dict(policy=mw.MW_ENGINE_POLLED, layers_per_launch=p, switch_on_decode_end=False),
    "polled_graph": lambda n_pl, p: dict(policy=mw.MW_ENGINE_POLLED, layers_per_launch=n_pl,
                                         switch_on_decode_end=False, decode_graph=True),
    "polled_switch_graph": lambda n_pl, p: dict(policy=mw.MW_ENGINE_POLLED, layers_per_launch=n_pl,
                                                switch_on_decode_end=True, decode_graph=True),
    "blocking_graph": lambda n_pl, p: dict(policy=mw.MW_ENGINE_BLOCKING, layers_per_launch=p,
                                           switch_on_decode_end=False, decode_graph=True),
}


def scenarios(L: int, args) -> Dict:
    """name -> (decode layers per iteration, decode iterations, prefill layers, variants).

    steady: decode iterations of N_T layers next to several N_T-layer prefill
        jobs; prefill ends first (the layer-wise overhead comparison).
    launch_bound: short decode iterations next to a prefill whose launch takes
        the host longer than one iteration runs (the paper's first bubble).
    decode_ends: decode finishes while most prefill layers remain (the
        paper's second bubble, removed by the switch)."""
    return {
        "steady": (L, args.decode_iters, L * args.prefill_batches,
                   ["blocking", "polled", "polled_switch", "polled_layer1", "polled_all", "polled_graph"]),
        "launch_bound": (2, 4 * args.decode_iters, L * args.prefill_batches,
                         ["blocking", "polled", "blocking_graph", "polled_graph"]),
        "decode_ends": (L, 2, 2 * L * args.prefill_batches, ["polled", "polled_switch", "polled_switch_graph"]),
    }


def write_table(out: Dict, path: str, argv):
    """Markdown summary of one measurement (the numbers the design notes use)."""
    cmd = "python -m paper_2504_14489_amd.engine " + " ".join(argv)
    g, dg = out["group"], out.get("decode_graphs", {})
    lines = [f"# Multiplex engine, workload {out['workload']} (N_T = {out['model_layers']} calls per decode iteration)",
             "", f"Command: `{cmd}`", "", f"N_PL from: {out['n_pl_from']}.", "",
             f"Partition group: {g['partitions']} partition(s) + whole-device stream, "
             f"{g['device_bytes'] / 2**20:.2f} MiB device memory, created in {g['create_ms']:.2f} ms.",
             f"Decode graphs: {dg.get('graphs', 0)}, {dg.get('device_bytes', 0) / 2**20:.2f} MiB, "
             f"{dg.get('capture_ms', 0.0):.2f} ms to capture, instantiate and upload.", ""]
    for p in out["partitions"]:
        lines += [f"## Prefill on {p['prefill_cus']} CUs (solo: decode call {p['decode_layer_ms']:.3f} ms, "
                  f"prefill call {p['prefill_layer_ms']:.3f} ms)", ""]
        if "estimate" in p:
            e = p["estimate"]
            lines += [f"Estimator (N_PL from it): prefill call {e['prefill_layer_ms_solo']:.3f} ms, decode call "
                      f"{e['decode_layer_ms_solo']:.3f} ms solo x guard {e['guard_slowdown']:.3f} = "
                      f"{e['decode_layer_ms_worst']:.3f} ms worst case.", ""]
        if "layerwise_overhead" in p:
            lines += [f"Layer-wise launch overhead on the prefill end, steady scenario: N_PL from the formula "
                      f"{100 * p['layerwise_overhead_npl']:+.2f}%, one layer per launch "
                      f"{100 * p['layerwise_overhead']:+.2f}% (both against the whole job in one launch).", ""]
        lines += [
                  "| scenario | variant | N_PL | wall ms | bubble % (decode / prefill) | decode iteration ms | "
                  "iteration gap us (median / max) | decode launch us | prefill end ms | switched layers | "
                  "switch: GPU gap / host us |", "|---|---|---|---|---|---|---|---|---|---|---|"]
        for sc_name, sc in p["scenarios"].items():
            for name, r in sc["runs"].items():
                sw = (f"{1e3 * r['switch_gap_ms']:.1f} / {r['switch_host_us']:.1f}"
                      if r["switch_gap_ms"] >= 0 else "-")
                lines.append(
                    f"| {sc_name} ({sc['decode_iters']} x {sc['decode_layers']} decode, {sc['prefill_layers']} prefill) "
                    f"| {name} | {r['n_pl_used']:.0f} | {r['wall_ms']:.2f} | {100 * r['bubble_ratio']:.2f} "
                    f"({100 * r['decode_bubble']:.2f} / {100 * r['prefill_bubble']:.2f}) | "
                    f"{r['decode_iter_ms_mean']:.3f} | {1e3 * r['iter_gap_ms_median']:.1f} / "
                    f"{1e3 * r['iter_gap_ms_max']:.1f} | {r['decode_launch_us_mean']:.0f} | {r['prefill_end_ms']:.2f} | "
                    f"{r['switched_layers']:.0f} | {sw} |")
        lines.append("")
    with open(path, "w") as f:
        f.write("\n".join(lines))


class Estimate:
    """The contention-tolerant estimator (paper Sec. 3.3) built from a profiling
    run (paper_2504_14489_amd.profiling --out): solo-run predictor fitted on the
    grid samples, contention guard over the measured pairs; worst case =
    solo prediction x guard slowdown."""

    def __init__(self, path: str):
        with open(path) as f:
            prof = json.load(f)
        self.model = prof["model"]
        self.p = mw.mw_predictor_create()
        self.g = mw.mw_guard_create()
        # prefill models over the simulated launch of the profiled shape
        mw.mw_predictor_set_launch_shape(self.p, self.model["num_q_heads"], self.model["num_kv_heads"])
        for smp in prof["prefill"]:
            if smp["grid"]:
                mw.mw_predictor_add_prefill(self.p, smp["cus"], [smp["n"]], [smp["r"]], smp["ms"])
        for smp in prof["decode"]:
            if smp["grid"]:
                mw.mw_predictor_add_decode(self.p, smp["cus"], smp["lens"], smp["ms"])
        mw.mw_predictor_fit(self.p)
        for smp in prof["pairs"]:
            if smp["slowdown"] is not None:
                mw.mw_guard_add(self.g, smp["prefill_new"], smp["prefill_reused"], smp["decode_batch"],
                                smp["decode_reused"], smp["prefill_cus"], smp["slowdown"])

    def layers(self, prefill_cus: int, new_lens, prefix_lens, dec_lens):
        """(solo prefill ms, solo decode ms, guard slowdown) of one prefill and
        one decode attention call on a prefill_cus / 256 - prefill_cus split."""
        t_p = mw.mw_predictor_prefill_ms(self.p, prefill_cus, new_lens, prefix_lens)
        t_d = mw.mw_predictor_decode_ms(self.p, 256 - prefill_cus, dec_lens)
        slow = mw.mw_guard_lookup(self.g, int(sum(new_lens)), int(sum(prefix_lens)), len(dec_lens),
                                  int(sum(int(L) - 1 for L in dec_lens)), prefill_cus)
        return t_p, t_d, slow

    def close(self):
        mw.mw_predictor_destroy(self.p)
        mw.mw_guard_destroy(self.g)


def main(argv=None):
    import torch
    from . import workloads as W
    from .device import DeviceWorkload, Timing

    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--config", default="llama8b")
    ap.add_argument("--prefill-cus", default="", help="comma list; default: the workload's partitions")
    ap.add_argument("--model-layers", type=int, default=32, help="N_T: attention calls per decode iteration")
    ap.add_argument("--decode-iters", type=int, default=12)
    ap.add_argument("--prefill-batches", type=int, default=4,
                    help="prefill jobs of N_T layers each, run back to back")
    ap.add_argument("--reps", type=int, default=3)
    ap.add_argument("--out", default="")
    ap.add_argument("--table", default="", help="also write a Markdown summary here")
    ap.add_argument("--scenarios", default="", help="comma list: run only these scenarios")
    ap.add_argument("--variants", default="", help="comma list: run only these variants")
    ap.add_argument("--profile", default="",
                    help="a profiling run's JSON: N_PL then comes from the estimator's worst-case latencies "
                         "instead of this run's solo measurements")
    argv = sys.argv[1:] if argv is None else list(argv)
    args = ap.parse_args(argv)

    cfg = W.CONFIGS[args.config]
    p_list = [int(x) for x in args.prefill_cus.split(",")] if args.prefill_cus else list(cfg.prefill_cus)
    wl = W.make_workload(cfg, seed=0)
    dw = DeviceWorkload(wl)
    dec, pre = dw.engine_args()
    L = args.model_layers
    out: Dict = {"workload": cfg.name, "model_layers": L, "partitions": []}
    est = None
    if args.profile:
        est = Estimate(args.profile)
        m = est.model
        if (m["num_q_heads"], m["num_kv_heads"], m["head_dim"]) != (cfg.hq, cfg.hkv, cfg.head_dim):
            raise SystemExit("the profile was taken for another model shape")
        out["n_pl_from"] = "estimator (solo-run prediction x contention guard)"
    else:
        out["n_pl_from"] = "solo latencies measured on the partition"

    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    eng = Engine(p_list)
    mem_bytes, create_ms = eng.memory()
    out["group"] = {"partitions": len(p_list), "device_bytes": mem_bytes, "create_ms": create_ms,
                    "device_bytes_seen_by_torch": free0 - torch.cuda.mem_get_info()[0]}
    log(f"[engine] group of {len(p_list)} partitions: {mem_bytes / 2**20:.2f} MiB, {create_ms:.2f} ms")

    # reference outputs of one call each, on the whole device (the decode
    # reference is taken again on each partition's decode stream below: the
    # balanced decode split depends on the stream's CU count, the prefill
    # result does not)
    whole_p, whole_d = eng.streams(-1)
    mw.mw_decode_attn(dec["pool"], dw.hq, dw.hkv, dw.d, dw.scale, dw.dec_lens, dec["d_seq_lens"],
                      dec["d_block_table"], dec["bt_stride"], dec["d_q"], dec["d_out"], dec["d_workspace"],
                      dec["workspace_bytes"], 0, whole_d, None)
    mw.mw_prefill_attn(pre["pool"], dw.hq, dw.hkv, dw.d, dw.scale, pre["new_lens"], pre["prefix_lens"],
                       pre["d_qo_indptr"], pre["d_prefix_lens"], pre["d_block_table"], pre["bt_stride"],
                       pre["d_q"], pre["d_out"], whole_p, None)
    mw.mw_sync(whole_p)
    ref_dec, ref_pre = dw.o_dec.clone(), dw.o_pre.clone()

    try:
        for ci, p_cus in enumerate(p_list):
            ps, ds = eng.streams(ci)
            # solo per-layer latencies on the partition -> N_PL (paper Sec. 3.4)
            td, tp = Timing(), Timing()
            for t, call in ((td, "d"), (tp, "p"), (td, "d"), (tp, "p")):
                if call == "d":
                    mw.mw_decode_attn(dec["pool"], dw.hq, dw.hkv, dw.d, dw.scale, dw.dec_lens, dec["d_seq_lens"],
                                      dec["d_block_table"], dec["bt_stride"], dec["d_q"], dec["d_out"],
                                      dec["d_workspace"], dec["workspace_bytes"], 0, ds, t.h)
                    mw.mw_sync(ds)
                else:
                    mw.mw_prefill_attn(pre["pool"], dw.hq, dw.hkv, dw.d, dw.scale, pre["new_lens"],
                                       pre["prefix_lens"], pre["d_qo_indptr"], pre["d_prefix_lens"],
                                       pre["d_block_table"], pre["bt_stride"], pre["d_q"], pre["d_out"], ps, t.h)
                    mw.mw_sync(ps)
            t_d, t_p = td.elapsed()[0], tp.elapsed()[0]
            ref_dec = dw.o_dec.clone()  # the solo decode calls ran on this partition's decode stream
            log(f"[engine] partition {p_cus}: decode layer {t_d:.3f} ms, prefill layer {t_p:.3f} ms")
            part = {"prefill_cus": p_cus, "decode_layer_ms": t_d, "prefill_layer_ms": t_p, "scenarios": {}}
            e_d, e_p = t_d, t_p
            if est is not None:
                sp, sd, slow = est.layers(p_cus, pre["new_lens"], pre["prefix_lens"], dw.dec_lens)
                # worst case: decode slowed by the guard; prefill at its solo prediction
                e_d, e_p = sd * slow, sp
                part["estimate"] = {"prefill_layer_ms_solo": sp, "decode_layer_ms_solo": sd, "guard_slowdown": slow,
                                    "decode_layer_ms_worst": e_d}
                log(f"[engine] estimator: prefill layer {sp:.3f} ms, decode layer {sd:.3f} ms x guard {slow:.3f}")
            for sc_name, (d_layers, d_iters, p_layers, variants) in scenarios(L, args).items():
                if args.scenarios and sc_name not in args.scenarios.split(","):
                    continue
                if args.variants:
                    variants = [v for v in variants if v in args.variants.split(",")]
                # N_PL = ceil(T_d * N_T / T_P) with the latencies of one decode
                # iteration and of one N_T-layer prefill job
                n_pl = mw.mw_prefill_layers(e_d * d_layers, e_p * L, L)
                sc = {"decode_layers": d_layers, "decode_iters": d_iters, "prefill_layers": p_layers,
                      "n_pl": n_pl, "runs": {}}
                for name in variants:
                    v = VARIANTS[name](n_pl, p_layers)
                    plan = dict(config=ci, decode_iters=d_iters, decode_layers=d_layers, prefill_layers=p_layers, **v)
                    eng.run(dec, pre, **plan)                     # warm-up
                    runs = [eng.run(dec, pre, **plan) for _ in range(args.reps)]
                    same = bool(torch.equal(ref_dec, dw.o_dec) and torch.equal(ref_pre, dw.o_pre))
                    st = _median_stats(runs)
                    st.update(gap_stats(eng.timeline(0), 1 if v.get("decode_graph") else d_layers))
                    st["outputs_equal_reference"] = same
                    st["n_pl_used"] = v["layers_per_launch"]
                    sc["runs"][name] = st
                    log(f"[engine] {p_cus:3d} CUs {sc_name:10s} {name:14s} wall {st['wall_ms']:7.2f} ms, "
                        f"bubble {100 * st['bubble_ratio']:5.2f}% (decode {100 * st['decode_bubble']:5.2f}%, "
                        f"prefill {100 * st['prefill_bubble']:5.2f}%), iter {st['decode_iter_ms_mean']:.3f} ms, "
                        f"iteration gap med/max {1e3 * st['iter_gap_ms_median']:.1f}/"
                        f"{1e3 * st['iter_gap_ms_max']:.1f} us, call gap med {1e3 * st['call_gap_ms_median']:.1f} us, "
                        f"prefill end {st['prefill_end_ms']:.2f} ms, switched {st['switched_layers']:.0f}, "
                        f"N_PL {v['layers_per_launch']}, host launch {st['host_launch_ms']:.2f} ms "
                        f"(decode iteration {st['decode_launch_us_mean']:.0f} us), same {same}")
                    if not same:
                        raise SystemExit("engine outputs differ from the reference call")
                part["scenarios"][sc_name] = sc
            r = part["scenarios"].get("steady", {}).get("runs", {})
            if all(k in r for k in ("polled_layer1", "polled_all", "polled")):
                part["layerwise_overhead"] = r["polled_layer1"]["prefill_end_ms"] / r["polled_all"]["prefill_end_ms"] - 1
                part["layerwise_overhead_npl"] = r["polled"]["prefill_end_ms"] / r["polled_all"]["prefill_end_ms"] - 1
            out["partitions"].append(part)
        n_g, g_bytes, g_ms = eng.graphs()
        out["decode_graphs"] = {"graphs": n_g, "device_bytes": g_bytes, "capture_ms": g_ms}
        log(f"[engine] {n_g} decode graphs: {g_bytes / 2**20:.2f} MiB, {g_ms:.1f} ms to capture")
    finally:
        eng.close()
        dw.close()
        if est is not None:
            est.close()
    line = json.dumps(out)
    print(line, flush=True)
    if args.out:
        with open(args.out, "w") as f:
            f.write(line + "\n")
    if args.table:
        write_table(out, args.table, argv)


if __name__ == "__main__":
    main()
