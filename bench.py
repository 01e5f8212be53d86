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
    args = ap.parse_args()
    if args.sources_hash:
        print(sources_hash())
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
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
