"""Drive a CPU build of libgemel's host code (stub HIP runtime, bounds-
checked launchers, AddressSanitizer) through one or more inference rounds of
a workload. Run as a subprocess with libasan preloaded; prints a JSON line
with the stub's counters."""

import ctypes
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from paper_2201_07705_amd import gemel as G  # noqa: E402
from workloads import configs  # noqa: E402


def stub_params(layers):
    """Parameter dicts of the shapes the workload generator makes, with
    constant values."""
    import numpy as np
    out = []
    for l in layers:
        if l["op"] not in ("conv", "fc"):
            out.append(None)
            continue
        shape = (l["cout"], l["cin"], l["kh"], l["kw"]) if l["op"] == "conv" \
            else (l["cout"], l["cin"])
        p = {"w": np.zeros(shape, np.float32), "b": None, "bn": None}
        if l["bias"]:
            p["b"] = np.zeros(l["cout"], np.float32)
        if l["bn"]:
            p["bn"] = (np.ones(l["cout"], np.float32),
                       np.zeros(l["cout"], np.float32),
                       np.zeros(l["cout"], np.float32),
                       np.ones(l["cout"], np.float32), 1e-5)
        out.append(p)
    return out


def main():
    libpath, name = sys.argv[1], sys.argv[2]
    kw = json.loads(sys.argv[3]) if len(sys.argv) > 3 else {}
    opts = json.loads(sys.argv[4]) if len(sys.argv) > 4 else {}
    rounds = int(sys.argv[5]) if len(sys.argv) > 5 else 2
    # per-round scenario: "streams" (stream index of each round), "capture"
    # (rounds enqueued while their stream reports an active capture),
    # "fail" ({round: n}: the n-th swap copy from that round on fails)
    scen = json.loads(sys.argv[6]) if len(sys.argv) > 6 else {}
    L = G.load(libpath)
    L.hipMalloc.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t]
    L.hipMalloc.restype = ctypes.c_int
    for f in ("hoststub_violations", "hoststub_launches", "hoststub_live_bytes",
              "hoststub_hazards", "hoststub_check_order", "hoststub_selftest",
              "hoststub_allocs", "hoststub_prefetches"):
        getattr(L, f).restype = ctypes.c_long
    L.hoststub_set_capturing.argtypes = [ctypes.c_void_p]
    L.hoststub_set_capturing.restype = None
    L.hoststub_last.restype = ctypes.c_char_p
    if name == "variants":   # every candidate group merged (tests/test_gpu_merging.py)
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        from test_gpu_merging import _variants_workload
        wl = _variants_workload(**kw)
    elif name == "many":     # more merged members than a launch holds (tests/test_gpu_merging.py)
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        from test_gpu_merging import _many_tiny
        wl = _many_tiny(kw.get("n", 18), kw.get("dtype", "bf16"))
    elif name == "chain":    # a deep unmerged chain (tests/test_gpu_layers.py)
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        from test_gpu_layers import _deep_chain
        from workloads.configs import ModelSpec, Workload
        wl = Workload("chain", 11, "bf16",
                      [ModelSpec("m0", "custom",
                                 _deep_chain(with_route=kw.get("route", True)),
                                 kw.get("frames", 3), (3, 24, 24))],
                      [], "uniform", options={"PAIRED_ACTS": 1})
    elif name == "grouped":  # one unmerged conv in several models (tests/test_gpu_layers.py)
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        from test_gpu_layers import GROUP_CASES, conv
        from workloads.configs import ModelSpec, Workload
        cin, cout, k, s_, p_, hw, frames = GROUP_CASES[kw.get("case", 0)]
        wl = Workload("grouped", 13, "bf16",
                      [ModelSpec(f"m{i}", "custom",
                                 [conv("c", -1, cin, cout, k, s_, p_, bn=True,
                                       act="leaky", out=True)], n, (cin, hw, hw))
                       for i, n in enumerate(frames)], [], "normal")
    else:
        wl = configs.get(name, **kw)
    # the stub computes nothing: constant parameters of the right shapes
    # (generating the seeded ones dominated the run time of large workloads)
    params = [stub_params(m.layers) for m in wl.models]

    def dev(nbytes):
        p = ctypes.c_void_p()
        assert L.hipMalloc(ctypes.byref(p), max(nbytes, 1)) == 0
        return p.value

    def one(scen):
        """One context through `rounds` rounds of scenario `scen`."""
        ctx = G.Context(0, wl.dtype, 0, library=L)
        ids = [ctx.register_model(m.layers, params[i], m.in_chw)
               for i, m in enumerate(wl.models)]
        ctx.merge([[(ids[a], b) for a, b in g] for g in wl.groups])
        if wl.budget_frac:
            ctx.set_option(G.OPT_WEIGHT_BUDGET,
                           int(wl.budget_frac * ctx.query(G.Q_UNMERGED_BYTES)))
        for k, v in wl.options.items():
            ctx.set_option(getattr(G, "OPT_" + k.upper()), int(v))
        for k, v in opts.items():
            ctx.set_option(getattr(G, k), v)
        frames, nfr, outs, outs_of = [], [], [], []
        for i, m in enumerate(wl.models):
            c, h, w = m.in_chw
            frames.append(dev(m.n_frames * c * h * w * 4))
            nfr.append(m.n_frames)
            outs_of.append([])
            for o in range(ctx.n_outputs(ids[i])):
                shp = ctx.output_shape(ids[i], o, m.n_frames)
                n = 1
                for d in shp:
                    n *= d
                outs_of[-1].append(dev(n * 4))
                outs.append(outs_of[-1][-1])
        # any non-null handles: enable graphs and streams
        streams = [dev(16) for _ in range(1 + max(scen.get("streams", [0])))]
        status, launches, round_allocs, cache = [], [], [], []
        subsets = scen.get("rounds")   # model indices of each round
        live_before = L.hoststub_live_bytes()
        allocs_before = L.hoststub_allocs()
        profile = None
        if "profile" in scen:   # measured cost table, then the rounds
            nb, reps = scen["profile"]
            pid = (ctypes.c_int32 * len(ids))(*ids)
            table = (ctypes.c_double * (len(ids) * nb))()
            st = L.gemel_profile_batches(ctx._h, pid, len(ids), nb, reps,
                                         streams[0], table)
            profile = {"status": st, "table": list(table),
                       "plans_after": ctx.query(G.Q_LAUNCHES),
                       "error": L.gemel_last_error(ctx._h).decode()}
        for r in range(rounds):
            st = streams[scen["streams"][r]] if "streams" in scen else streams[0]
            if str(r) in scen.get("fail", {}):
                ctx.set_option(G.OPT_FAIL_COPY_AT, scen["fail"][str(r)])
            if str(r) in scen.get("fail_alloc", {}):
                ctx.set_option(G.OPT_FAIL_ALLOC_AT, scen["fail_alloc"][str(r)])
            cap = r in scen.get("capture", [])
            if cap:
                L.hoststub_set_capturing(st)
            before = L.hoststub_launches()
            a_before = L.hoststub_allocs()
            if subsets is not None:
                sub = subsets[r]
                if scen.get("next", True):
                    ctx.set_next_round([ids[i] for i in subsets[r + 1]]
                                       if r + 1 < len(subsets) else [])
                status.append(ctx.infer_raw(
                    [ids[i] for i in sub], [frames[i] for i in sub],
                    [nfr[i] for i in sub], [p for i in sub for p in outs_of[i]],
                    st))
                cache.append([ctx.query(G.Q_ROUND_LOADED_BYTES),
                              ctx.query(G.Q_ROUND_EVICTED_BYTES),
                              ctx.query(G.Q_CACHED_BYTES)])
            else:
                status.append(ctx.infer_raw(ids, frames, nfr, outs, st,
                                            noalloc=r in scen.get("noalloc", [])))
            launches.append(L.hoststub_launches() - before)
            round_allocs.append(L.hoststub_allocs() - a_before)
            if cap:
                L.hoststub_set_capturing(None)
        L.hoststub_check_order()
        res = {
            "status": status,
            "round_launches": launches,
            "round_allocs": round_allocs,
            "cache": cache,
            "cache_capacity": ctx.query(G.Q_CACHE_CAPACITY),
            "load_order": ctx.load_order(ids),
            "allocs": L.hoststub_allocs() - allocs_before,
            "error": L.gemel_last_error(ctx._h).decode(),
            "plan_launches": ctx.query(G.Q_LAUNCHES),
            "plan_prefetches": ctx.query(G.Q_PREFETCHES),
            "arena": ctx.query(G.Q_ACTIVATION_BYTES),
            "streamed": ctx.query(G.Q_STREAMED_BYTES),
            "round_mode": ctx.query(G.Q_ROUND_MODE),
            "profile": profile,
        }
        ctx.close()
        # device bytes the context still held after it was destroyed
        res["leaked"] = L.hoststub_live_bytes() - live_before
        return res

    def totals(res):
        return dict(res, **{
            "selftest": L.hoststub_selftest(),
            "hazards": L.hoststub_hazards(),
            "violations": L.hoststub_violations(),
            "launches": L.hoststub_launches(),
            "prefetches": L.hoststub_prefetches(),
            "last": L.hoststub_last().decode(),
        })

    if "each" in scen:
        # several scenarios, each in a fresh context; counters accumulate
        runs = [one(sc) for sc in scen["each"]]
        print(json.dumps(totals({"runs": runs})), flush=True)
    else:
        print(json.dumps(totals(one(scen))), flush=True)


if __name__ == "__main__":
    main()
