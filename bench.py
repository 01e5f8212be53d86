#!/usr/bin/env python3
"""Merged multi-model inference throughput on one MI355X.

One step is one inference round of a merged workload: every model's frame
batch goes through the whole hot path (input pack, merged and per-model
convs with fused epilogues, pools, routing, FC heads, fp32 outputs) in one
gemel_infer call, inputs already resident in HBM. The default workload is
two ResNet-50 sharing stem + layer1..3 and two VGG-16 sharing all convs, 8
frames each at 3x224x224 (the ResNet-50 configuration named by the
throughput target); --config selects any other workload.

Prints one JSON line: whole-job frames/s, ms per step, the roofline of the
dominant kernel family (HIP-event timings collected by the library with
profiling on, in separate passes after the timed region: one stream for
`roofline`, the round's streams for `roofline_concurrent`), its HBM traffic
per launch from the committed counter summary, and the CPU oracle timed on
a bounded sample of the same workload.
"""

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("merged multi-model frames/sec on 1 GPU; conv TFLOP/s as % of "
          "bf16 MFMA peak")
PEAK_BF16_TFLOPS = 2516.6   # 256 CU x 4096 FLOP/clk x 2.4 GHz, dense
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0

DESCRIPTIONS = {
    "tiny2": "2 tiny CNNs sharing 2 convs, fp32, 1 frame each, 3x32x32",
    "resnet18x2": "2x ResNet-18, all convs merged, 4 frames each, 3x224x224",
    "r50x2_vgg16x2": "2x ResNet-50 (stem+layer1-3 merged) + 2x VGG-16 "
                     "(13 convs merged), 8 frames each, 3x224x224",
    "yolov3x3": "3x YOLOv3 sharing the Darknet-53 backbone, 4 frames each, "
                "3x416x416",
    "mix8_budget40": "ResNet-152x2 + ResNet-50x3 + VGG-19x3, partial "
                     "merging, 8 frames each, 3x224x224, weights capped at "
                     "40% of the unmerged bytes (rest streamed per round)",
}


# HBM traffic of the conv family per launch, from two rocprofv3 --pmc runs of
# this script (FETCH_SIZE, WRITE_SIZE) scaled by what the same counters read
# for a plain device copy of known size (--calibrate-copy). The summary
# records a hash of the sources that decide the conv kernels and their
# launch shapes; the figure is reported only while they are unchanged.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_conv_r50x2_vgg16x2.md")
TRAFFIC_SOURCES = ["k_conv.hip", "k_conv_dma.hip", "k_stem.hip", "kernels.h",
                   "kargs.h", "conv_epi.h", "splitk.h", "plan.cpp"]


def sources_hash():
    h = hashlib.sha256()
    for f in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, "paper_2201_07705_amd", "csrc", f),
                  "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def recorded_traffic(workload, kernel):
    """Bytes per launch from the committed counter summary, or None."""
    try:
        text = open(TRAFFIC_FILE).read()
    except OSError:
        return None
    m = re.search(r"<!-- traffic: (\{.*?\}) -->", text)
    if not m:
        return None
    rec = json.loads(m.group(1))
    if (rec.get("workload") != workload or rec.get("kernel") != kernel
            or rec.get("sources_sha256") != sources_hash()):
        return None
    return rec.get("bytes_per_launch")


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr,
          flush=True)


def cpu_baseline(wl, params, frames, seconds):
    """The oracle (test infrastructure) on the host cores, on a bounded
    sample: frame j of every model, j = 0, 1, ... until `seconds` pass."""
    import oracle
    from oracle import model as om
    eff = om.effective_params(params, wl.groups)
    done, t0, j = 0, time.perf_counter(), 0
    max_n = max(m.n_frames for m in wl.models)
    while j < max_n:
        for i, m in enumerate(wl.models):
            if j < m.n_frames:
                om.run_model(m.layers, eff[i], frames[i][j:j + 1])
                done += 1
        j += 1
        if time.perf_counter() - t0 >= seconds:
            break
    dt = time.perf_counter() - t0
    return {"value": done / dt, "unit": "frames/s",
            "cores": oracle.threads(), "kind": "oracle",
            "sample": f"{done} frames ({j} per model) of the same workload, "
                      f"{dt:.1f} s, fp32 with fp64 accumulation"}


def run_workload(wl, args, options, G, P, torch, steps, warmup,
                 profile_steps):
    """Register, merge and time one workload; returns the measurements."""
    log(f"workload {wl.name}: generating seeded inputs")
    params = [wl.params(i) for i in range(len(wl.models))]
    frames = [wl.frames(i) for i in range(len(wl.models))]
    ctx = P.Context(0, wl.dtype)
    ids = [ctx.register_model(m.layers, params[i], m.in_chw)
           for i, m in enumerate(wl.models)]
    ctx.merge([[(ids[a], b) for a, b in g] for g in wl.groups])
    opts = dict(wl.options)
    opts.update(options)
    for name, value in opts.items():
        ctx.set_option(getattr(G, "OPT_" + name.upper()), int(value))
    budget = 0
    if wl.budget_frac:
        budget = int(wl.budget_frac * ctx.query(G.Q_UNMERGED_BYTES))
        ctx.set_option(G.OPT_WEIGHT_BUDGET, budget)
    dev = [torch.from_numpy(f).cuda() for f in frames]
    stream = torch.cuda.Stream()
    outs = ctx.alloc_outputs(ids, [m.n_frames for m in wl.models])
    log(f"warmup {warmup}")
    with torch.cuda.stream(stream):
        for _ in range(warmup):
            ctx.infer(ids, dev, stream=stream, outputs=outs)
        # the round-mode tuner times its candidates over the first rounds
        # of a plan: the timed region starts once its choice is fixed,
        # whatever the warmup count
        extra = 0
        while ctx.query(G.Q_ROUND_TUNING) > 0:
            ctx.infer(ids, dev, stream=stream, outputs=outs)
            extra += 1
    torch.cuda.synchronize()
    if extra:
        log(f"{extra} more warmup rounds until the round-mode tuner settled")
    log(f"timed {steps} steps")
    ev0, ev1 = torch.cuda.Event(enable_timing=True), \
        torch.cuda.Event(enable_timing=True)
    # record both events once so that their lazy creation (which can stall
    # the host for tens of milliseconds) happens outside the timed region
    with torch.cuda.stream(stream):
        ev0.record(stream)
        ev1.record(stream)
    torch.cuda.synchronize()
    tuning_before = ctx.query(G.Q_ROUND_TUNING)
    t0 = time.perf_counter()
    with torch.cuda.stream(stream):
        ev0.record(stream)
        for _ in range(steps):
            ctx.infer(ids, dev, stream=stream, outputs=outs)
        ev1.record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    wall_s = t1 - t0
    ev_ms = ev0.elapsed_time(ev1)
    step_ms = wall_s * 1e3 / steps
    fps = wl.total_frames() * steps / wall_s
    flops = wl.flops()
    streamed = ctx.query(G.Q_STREAMED_BYTES)
    launches = ctx.query(G.Q_LAUNCHES)
    round_mode = ["enqueue", "stream_segments", "data_graph", "stream_graph",
                  "serial"][ctx.query(G.Q_ROUND_MODE)]

    # per-kernel-family HIP-event timings (separate, untimed passes): on one
    # stream (each kernel alone on the GPU: the roofline figure, comparable
    # with the counter runs, which serialise dispatches) and with the round's
    # streams, as in the timed region (kernels share the GPU, and a launch's
    # start event also counts its wait for compute units)
    def profiled(streams):
        log(f"profiled pass {profile_steps} steps, {streams} stream(s)")
        saved = ctx.query(G.Q_STREAMS)
        ctx.set_option(G.OPT_STREAMS, streams)
        ctx.set_option(G.OPT_PROFILE, 1)
        with torch.cuda.stream(stream):
            for _ in range(profile_steps):
                ctx.infer(ids, dev, stream=stream, outputs=outs)
        torch.cuda.synchronize()
        pr, _ = ctx.profile()
        ctx.set_option(G.OPT_PROFILE, 0)
        ctx.set_option(G.OPT_STREAMS, saved)
        return pr

    prof = profiled(ctx.query(G.Q_STREAMS))
    prof1 = profiled(1)
    # the dominant family (conv_merged is a subset of conv_mfma)
    fam = max((k for k in prof1 if k != "conv_merged"),
              key=lambda k: prof1[k]["ms"])

    def roofline(pr, fam):
        st = pr[fam]
        if fam in ("conv_mfma", "conv_merged", "conv_f32") or (
                fam == "fc" and st["flops"] / st["bytes"] > 315):
            peak = PEAK_BF16_TFLOPS if wl.bf16 else PEAK_FP32_TFLOPS
            ach = st["flops"] / (st["ms"] * 1e-3) / 1e12
            r = {"bound": "mfma" if wl.bf16 else "alu", "achieved": ach,
                 "peak": peak, "unit": "TFLOP/s", "frac": ach / peak}
        else:
            ach = st["bytes"] / (st["ms"] * 1e-3) / 1e9
            r = {"bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS,
                 "unit": "GB/s", "frac": ach / PEAK_HBM_GBS}
        r.update({"kernel": fam, "launches_per_step": st["launches"],
                  "avg_launch_us": st["ms"] * 1e3 / max(st["launches"], 1),
                  "algorithmic_per_launch":
                      (st["flops"] if r["unit"] == "TFLOP/s" else
                       st["bytes"]) / max(st["launches"], 1)})
        return r

    roof = roofline(prof1, fam)
    roof["traffic"] = recorded_traffic(wl.name, fam)
    roof_conc = roofline(prof, fam)
    merged = None
    if prof1.get("conv_merged", {}).get("launches"):
        merged = roofline(prof1, "conv_merged")
    kern = {}
    for k, v in prof1.items():
        if v["launches"]:
            kern[k] = {"launches": v["launches"], "ms": round(v["ms"], 4),
                       "tflops": round(v["flops"] / v["ms"] / 1e9, 2)
                       if v["ms"] and v["flops"] else None,
                       "gbs": round(v["bytes"] / v["ms"] / 1e6, 1)
                       if v["ms"] else None}
    ctx.close()
    return {
        "wl": wl, "params": params, "frames": frames, "fps": fps,
        "step_ms": step_ms, "ev_ms": ev_ms, "flops": flops,
        "budget": budget, "streamed": streamed, "launches": launches,
        "round_mode": round_mode, "roof": roof, "roof_conc": roof_conc,
        "merged": merged, "kern": kern, "options": opts,
        "tuning_in_timed": min(tuning_before, steps),
    }


def host_link_gbs(torch, mib=256, reps=10):
    """Pinned host to device copy rate (GB/s) of one large transfer."""
    src = torch.empty(mib << 20, dtype=torch.uint8).pin_memory()
    dst = torch.empty(mib << 20, dtype=torch.uint8, device="cuda")
    for _ in range(2):
        dst.copy_(src, non_blocking=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        dst.copy_(src, non_blocking=True)
    torch.cuda.synchronize()
    return reps * (mib << 20) / (time.perf_counter() - t0) / 1e9


def swap_leg(wl, G, P, torch, steps):
    """Weight swapping on a budget (Section 3.2; Section 5.4 and Appendix
    A.4 for the weight cache): round times with swapping against the same
    rounds with every weight resident, the bytes each round copies, and the
    ideal round time max(resident round, bytes / measured host-link rate)
    that perfect overlap of copies and compute would reach. How much of
    the copies actually overlaps kernels comes from a trace
    (--trace-summary)."""
    log(f"swap leg on {wl.name}: seeded inputs")
    params = [wl.params(i) for i in range(len(wl.models))]
    frames = [wl.frames(i) for i in range(len(wl.models))]
    dev = [torch.from_numpy(f).cuda() for f in frames]
    rate = host_link_gbs(torch)
    log(f"host link {rate:.1f} GB/s")

    def context(opts):
        ctx = P.Context(0, wl.dtype)
        ids = [ctx.register_model(m.layers, params[i], m.in_chw)
               for i, m in enumerate(wl.models)]
        ctx.merge([[(ids[a], b) for a, b in g] for g in wl.groups])
        for k, v in dict(wl.options, **opts).items():
            ctx.set_option(getattr(G, "OPT_" + k.upper()), int(v))
        return ctx, ids

    def timed(ctx, ids, rounds, reps):
        """ms per round of the round list (model index lists), after two
        untimed passes; loaded bytes per round of the last pass."""
        stream = torch.cuda.Stream()
        outs = {i: ctx.alloc_outputs([ids[i]], [wl.models[i].n_frames])[0]
                for i in range(len(ids))}

        def one_pass(record):
            loaded = []
            for r, sub in enumerate(rounds):
                nxt = rounds[(r + 1) % len(rounds)]
                if ctx.query(G.Q_CACHE_CAPACITY):
                    ctx.set_next_round([ids[i] for i in nxt])
                ctx.infer([ids[i] for i in sub], [dev[i] for i in sub],
                          stream=stream, outputs=[outs[i] for i in sub])
                if record:
                    loaded.append(ctx.query(G.Q_ROUND_LOADED_BYTES))
            return loaded
        with torch.cuda.stream(stream):
            for _ in range(2):
                one_pass(False)
            while ctx.query(G.Q_ROUND_TUNING) > 0:
                one_pass(False)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        loaded = []
        with torch.cuda.stream(stream):
            for _ in range(reps):
                loaded = one_pass(True)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3 / (reps * len(rounds)), loaded

    out = {"workload": wl.name, "host_link_gbs": rate}
    all_models = [list(range(len(wl.models)))]
    # streaming: every model in one round, the budget's non-resident
    # weights copied through the staging slots every round
    ctx, ids = context({})
    unmerged = ctx.query(G.Q_UNMERGED_BYTES)
    budget = int(wl.budget_frac * unmerged)
    ctx.close()
    ctx, ids = context({"WEIGHT_BUDGET": budget})
    ms_s, _ = timed(ctx, ids, all_models, steps)
    streamed = ctx.query(G.Q_STREAMED_BYTES)
    ctx.close()
    ctx, ids = context({})
    ms_r, _ = timed(ctx, ids, all_models, steps)
    ctx.close()
    copy_ms = streamed / rate / 1e6
    out["streaming"] = {
        "budget_bytes": budget, "round_ms": ms_s, "resident_round_ms": ms_r,
        "copied_bytes_per_round": streamed, "copy_ms_at_link_rate": copy_ms,
        "ideal_round_ms": max(ms_r, copy_ms),
        "frames_per_s": wl.total_frames() / ms_s * 1e3}
    log(f"streaming {ms_s:.2f} ms/round vs resident {ms_r:.2f}, "
        f"{streamed / 1e6:.0f} MB copied")
    # weight cache: round-robin rounds over subsets in the library's
    # sharing-aware load order; the budget grows by quarters from the
    # streaming one until the rounds' pinned weights fit the cache
    for per in (1, 2):
        b = budget
        while True:
            ctx, ids = context({"WEIGHT_BUDGET": b, "SWAP_CACHE": 1})
            order = ctx.load_order(ids)
            idx = [ids.index(i) for i in order]
            rounds = [idx[i:i + per] for i in range(0, len(idx), per)]
            try:
                ms_c, loaded = timed(ctx, ids, rounds, max(2, steps // 10))
                cap = ctx.query(G.Q_CACHE_CAPACITY)
                ctx.close()
                break
            except G.GemelError as e:
                ctx.close()
                if e.code != G.EBUDGET or b > 4 * budget:
                    raise
                b = b * 5 // 4
        ctx, ids = context({})
        ms_rr, _ = timed(ctx, ids, rounds, max(2, steps // 10))
        ctx.close()
        lb = sum(loaded) / len(loaded)
        cms = lb / rate / 1e6
        out[f"cache_{per}_per_round"] = {
            "budget_bytes": b, "cache_bytes": cap, "rounds_per_cycle": len(rounds),
            "round_ms": ms_c, "resident_round_ms": ms_rr,
            "loaded_bytes_per_round": lb, "copy_ms_at_link_rate": cms,
            "ideal_round_ms": max(ms_rr, cms)}
        log(f"cache, {per} model(s) per round: {ms_c:.2f} ms/round vs "
            f"resident {ms_rr:.2f}, {lb / 1e6:.0f} MB loaded per round")
    return out


def trace_summary(path, gap_ms=50.0):
    """Copy/compute overlap from a rocprofv3 CSV trace directory (kernel and
    memory-copy traces): the run is cut into phases at idle gaps longer
    than gap_ms; per phase, host-to-device copy count, bytes unknown to the
    trace, busy time of the copy engine and of the kernels, and the time
    both were busy (the copy time hidden behind compute)."""
    import csv
    import glob

    def intervals(pattern, pred):
        out = []
        for f in glob.glob(os.path.join(path, pattern)):
            for r in csv.DictReader(open(f)):
                if pred(r):
                    out.append((int(r["Start_Timestamp"]),
                                int(r["End_Timestamp"])))
        return sorted(out)

    def union(iv):
        out = []
        for a, b in iv:
            if out and a <= out[-1][1]:
                out[-1][1] = max(out[-1][1], b)
            else:
                out.append([a, b])
        return out

    def length(u):
        return sum(b - a for a, b in u)

    def inter(u, v):
        i = j = 0
        t = 0
        while i < len(u) and j < len(v):
            a, b = max(u[i][0], v[j][0]), min(u[i][1], v[j][1])
            t += max(0, b - a)
            if u[i][1] < v[j][1]:
                i += 1
            else:
                j += 1
        return t

    cp = intervals("*memory_copy_trace.csv",
                   lambda r: "HOST_TO_DEVICE" in r.get("Direction", ""))
    kn = intervals("*kernel_trace.csv", lambda r: True)
    everything = union(sorted(cp + kn))
    phases = [[everything[0][0], everything[0][1]]]
    for a, b in everything[1:]:
        if a - phases[-1][1] > gap_ms * 1e6:
            phases.append([a, b])
        else:
            phases[-1][1] = b
    rows = []
    for a, b in phases:
        c = union([x for x in cp if a <= x[0] < b])
        k = union([x for x in kn if a <= x[0] < b])
        if not c:
            continue
        rows.append({"span_ms": (b - a) / 1e6, "copies": sum(1 for x in cp if a <= x[0] < b),
                     "copy_busy_ms": length(c) / 1e6, "kernel_busy_ms": length(k) / 1e6,
                     "copy_hidden_ms": inter(c, k) / 1e6,
                     "copy_hidden_fraction": inter(c, k) / max(1, length(c))})
    return rows


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="r50x2_vgg16x2",
                    choices=sorted(DESCRIPTIONS))
    ap.add_argument("--also", default="yolov3x3",
                    help="second workload measured in the same run and "
                         "reported under 'also' (the other configuration "
                         "the conv target is quoted on); 'none' to skip")
    ap.add_argument("--also-steps", type=int, default=100)
    ap.add_argument("--swap", default="mix8_budget40",
                    help="workload with a weight budget measured under "
                         "'swap' (streaming every round, and the weight "
                         "cache over one- and two-model rounds); 'none' to "
                         "skip")
    ap.add_argument("--swap-steps", type=int, default=20)
    ap.add_argument("--profile-steps", type=int, default=20)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only copy MIB MiB device to device once (the "
                         "reference kernel for byte-counter scaling)")
    ap.add_argument("--option", action="append", default=[],
                    metavar="NAME=VALUE",
                    help="library option set before the first round, e.g. "
                         "SPLITK_FUSED=0 (repeatable)")
    ap.add_argument("--sources-hash", action="store_true",
                    help="print the hash recorded with traffic figures")
    ap.add_argument("--trace-summary", metavar="DIR",
                    help="only summarise copy/compute overlap of a rocprofv3 "
                         "CSV trace directory (kernel and memory-copy "
                         "traces), one JSON line per phase")
    args = ap.parse_args()
    if args.sources_hash:
        print(sources_hash())
        return
    if args.trace_summary:
        for row in trace_summary(args.trace_summary):
            print(json.dumps(row))
        return
    if args.calibrate_copy:
        import torch
        n = args.calibrate_copy << 18          # float32 elements
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n * 4}))
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): "
              "merged inference keeps each merged group's weights on one "
              "device and needs no collectives", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2201_07705_amd as P
    from paper_2201_07705_amd import gemel as G
    from workloads import configs

    options = {}
    for o in args.option:
        name, _, value = o.partition("=")
        options[name.upper()] = int(value)
    main_r = run_workload(configs.get(args.config), args, options, G, P,
                          torch, args.steps, args.warmup, args.profile_steps)
    wl = main_r["wl"]
    also = None
    if args.also != "none" and args.also != args.config:
        a = run_workload(configs.get(args.also), args, options, G, P, torch,
                         args.also_steps, args.warmup, args.profile_steps)
        also = {
            "workload": a["wl"].name, "description": DESCRIPTIONS[a["wl"].name],
            "frames_per_s": a["fps"], "ms_per_step": a["step_ms"],
            "steps": args.also_steps, "frames_per_step": a["wl"].total_frames(),
            "tflops_per_step": a["flops"] / (a["step_ms"] * 1e-3) / 1e12,
            "roofline": a["roof"], "roofline_merged_conv": a["merged"],
            "round_mode": a["round_mode"], "options": a["options"],
            "tuning_rounds_in_timed_region": a["tuning_in_timed"],
            "kernels": a["kern"],
        }

    swap = None
    if args.swap != "none":
        swap = swap_leg(configs.get(args.swap), G, P, torch, args.swap_steps)

    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle on host cores)")
        cpu = cpu_baseline(wl, main_r["params"], main_r["frames"],
                           args.cpu_seconds)

    line = {
        "metric": METRIC, "value": main_r["fps"], "unit": "frames/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": main_r["step_ms"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if wl.bf16 else "f32", "data": "synthetic",
        "config": {"workload": wl.name, "description": DESCRIPTIONS[wl.name],
                   "frames_per_step": wl.total_frames(),
                   "gflop_per_step": round(main_r["flops"] / 1e9, 2),
                   "merged_groups": len(wl.groups),
                   "weight_budget_bytes": main_r["budget"]},
        "tflops_per_step": main_r["flops"] / (main_r["step_ms"] * 1e-3) / 1e12,
        "event_ms_per_step": main_r["ev_ms"] / args.steps,
        "tuning_rounds_in_timed_region": main_r["tuning_in_timed"],
        "roofline": main_r["roof"],
        "roofline_merged_conv": main_r["merged"],
        "roofline_concurrent": main_r["roof_conc"], "kernels": main_r["kern"],
        "cpu_baseline": cpu,
        "round_mode": main_r["round_mode"],
        "streamed_bytes_per_step": main_r["streamed"],
        "launches_per_step": main_r["launches"],
        "options": main_r["options"],
        "also": also,
        "swap": swap,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
