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


def main():
    libpath, name = sys.argv[1], sys.argv[2]
    kw = json.loads(sys.argv[3]) if len(sys.argv) > 3 else {}
    opts = json.loads(sys.argv[4]) if len(sys.argv) > 4 else {}
    rounds = int(sys.argv[5]) if len(sys.argv) > 5 else 2
    L = G.load(libpath)
    L.hipMalloc.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t]
    L.hipMalloc.restype = ctypes.c_int
    for f in ("hoststub_violations", "hoststub_launches", "hoststub_live_bytes",
              "hoststub_hazards", "hoststub_check_order", "hoststub_selftest"):
        getattr(L, f).restype = ctypes.c_long
    L.hoststub_last.restype = ctypes.c_char_p
    if name == "variants":   # every candidate group merged (tests/test_gpu_merging.py)
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        from test_gpu_merging import _variants_workload
        wl = _variants_workload(**kw)
    else:
        wl = configs.get(name, **kw)
    ctx = G.Context(0, wl.dtype, 0, library=L)
    ids = [ctx.register_model(m.layers, wl.params(i), m.in_chw)
           for i, m in enumerate(wl.models)]
    ctx.merge([[(ids[a], b) for a, b in g] for g in wl.groups])
    if wl.budget_frac:
        ctx.set_option(G.OPT_WEIGHT_BUDGET,
                       int(wl.budget_frac * ctx.query(G.Q_UNMERGED_BYTES)))
    for k, v in opts.items():
        ctx.set_option(getattr(G, k), v)

    def dev(nbytes):
        p = ctypes.c_void_p()
        assert L.hipMalloc(ctypes.byref(p), max(nbytes, 1)) == 0
        return p.value

    frames, nfr, outs = [], [], []
    for i, m in enumerate(wl.models):
        c, h, w = m.in_chw
        frames.append(dev(m.n_frames * c * h * w * 4))
        nfr.append(m.n_frames)
        for o in range(ctx.n_outputs(ids[i])):
            shp = ctx.output_shape(ids[i], o, m.n_frames)
            n = 1
            for d in shp:
                n *= d
            outs.append(dev(n * 4))
    stream = dev(16)   # any non-null handle: enables graphs and streams
    status = []
    for _ in range(rounds):
        status.append(ctx.infer_raw(ids, frames, nfr, outs, stream))
    L.hoststub_check_order()
    print(json.dumps({
        "selftest": L.hoststub_selftest(),
        "hazards": L.hoststub_hazards(),
        "status": status,
        "violations": L.hoststub_violations(),
        "launches": L.hoststub_launches(),
        "last": L.hoststub_last().decode(),
        "plan_launches": ctx.query(G.Q_LAUNCHES),
        "arena": ctx.query(G.Q_ACTIVATION_BYTES),
        "streamed": ctx.query(G.Q_STREAMED_BYTES),
        "error": L.gemel_last_error(ctx._h).decode(),
    }), flush=True)
    ctx.close()


if __name__ == "__main__":
    main()
