"""ctypes binding of libgemel (include/gemel.h): the same entry points,
argument marshalling only. Every layer of every model runs in the HIP
kernels of libgemel.so; there is no Python or CPU fallback: importing this
module without the built library raises.

``Context`` wraps the calls for Python callers: layers are given as dicts
(op, src0, src1, cin, cout, kh, kw, stride, pad, act, res, res_mode, out;
see workloads/zoo.py for the format) with per-layer parameter dicts
(w, b, bn = (gamma, beta, mean, var, eps)); device buffers and streams come
from torch.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgemel.so")

# status codes
OK, EINVAL, ENOMEM, ESHAPE, ENOTMERGEABLE, EBUDGET, EDEVICE, ESTATE = \
    0, -1, -2, -3, -4, -5, -6, -7
STATUS_NAMES = {0: "OK", -1: "EINVAL", -2: "ENOMEM", -3: "ESHAPE",
                -4: "ENOTMERGEABLE", -5: "EBUDGET", -6: "EDEVICE",
                -7: "ESTATE"}
F32, BF16 = 0, 1
OP = {"conv": 0, "fc": 1, "maxpool": 2, "avgpool": 3, "upsample": 4,
      "concat": 5}
ACT = {"none": 0, "relu": 1, "leaky": 2}
RES_MODE = {"add_act": 0, "act_add": 1}
LEAKY_SLOPE = 0.1

Q_UNMERGED_BYTES, Q_MERGED_BYTES, Q_RESIDENT_BYTES, Q_PEAK_BYTES, \
    Q_STREAMED_BYTES, Q_ACTIVATION_BYTES, Q_LAUNCHES, Q_N_MODELS, \
    Q_GRAPH_REPLAYS, Q_STREAMS, Q_ROUND_MODE, Q_ROUND_TUNING, \
    Q_ROUND_LOADED_BYTES, Q_ROUND_EVICTED_BYTES, Q_CACHED_BYTES, \
    Q_CACHE_CAPACITY, Q_PREFETCHES = range(17)
OPT_USE_GRAPH, OPT_SWAP_SLOT_BYTES, OPT_SWAP_SLOTS, OPT_FAIL_COPY_AT, \
    OPT_SPLIT_MERGED, OPT_WEIGHT_BUDGET, OPT_PROFILE, OPT_CONV_TILE, \
    OPT_CONV_SPLITS, OPT_STREAMS, OPT_GRAPH_DAG, OPT_FORK_US, \
    OPT_AUTOTUNE, OPT_SPLITK_FUSED, OPT_TUNE, OPT_FUSE_POOL, \
    OPT_MIXED_SIZES, OPT_PAIRED_ACTS, OPT_FAIL_ALLOC_AT, \
    OPT_GROUP_UNMERGED, OPT_SWAP_CACHE, OPT_PREFETCH = range(22)
KERNEL_FAMILIES = ("conv_mfma", "conv_f32", "splitk_reduce", "fc", "pack",
                   "pool", "route", "export", "conv_merged")

EXPORTED = ("gemel_create", "gemel_register_model", "gemel_merge",
            "gemel_enumerate_groups", "gemel_infer", "gemel_infer_noalloc",
            "gemel_set_next_round", "gemel_load_order",
            "gemel_sla_batches", "gemel_profile_batches",
            "gemel_model_outputs", "gemel_output_shape",
            "gemel_query", "gemel_set_option", "gemel_profile",
            "gemel_last_error", "gemel_destroy")

_fp = ctypes.POINTER(ctypes.c_float)


class LayerDesc(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int32), ("src0", ctypes.c_int32),
                ("src1", ctypes.c_int32), ("cin", ctypes.c_int32),
                ("cout", ctypes.c_int32), ("kh", ctypes.c_int32),
                ("kw", ctypes.c_int32), ("stride", ctypes.c_int32),
                ("pad", ctypes.c_int32), ("act", ctypes.c_int32),
                ("act_slope", ctypes.c_float), ("res_src", ctypes.c_int32),
                ("res_mode", ctypes.c_int32), ("is_output", ctypes.c_int32),
                ("weight", _fp), ("bias", _fp), ("bn_gamma", _fp),
                ("bn_beta", _fp), ("bn_mean", _fp), ("bn_var", _fp),
                ("bn_eps", ctypes.c_float)]


class Member(ctypes.Structure):
    _fields_ = [("model_id", ctypes.c_int32), ("layer", ctypes.c_int32)]


class Group(ctypes.Structure):
    _fields_ = [("n_members", ctypes.c_int32),
                ("members", ctypes.POINTER(Member))]


class KernelStat(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("launches", ctypes.c_int32),
                ("flops", ctypes.c_double), ("bytes", ctypes.c_double),
                ("ms", ctypes.c_double)]


class GemelError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {msg}")
        self.code = code


_lib = None


def _hip_runtimes():
    """Paths of every HIP runtime library mapped into this process."""
    paths = set()
    try:
        with open("/proc/self/maps") as f:
            for line in f:
                if "libamdhip64" in line:
                    paths.add(os.path.realpath(line.split()[-1]))
    except OSError:
        pass
    return paths


def load(path):
    """Load another build of the same ABI (e.g. a CPU build of the host
    code used by the tests) with its C signatures declared."""
    return _configure(ctypes.CDLL(path))


def _configure(L):
    """Declare the C signatures of the ABI on a loaded library."""
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    L.gemel_create.argtypes = [ctypes.POINTER(vp), i32, i32,
                               ctypes.c_uint64]
    L.gemel_register_model.argtypes = [vp, ctypes.POINTER(LayerDesc), i32,
                                       i32, i32, i32,
                                       ctypes.POINTER(i32)]
    L.gemel_merge.argtypes = [vp, ctypes.POINTER(Group), i32]
    L.gemel_enumerate_groups.argtypes = [
        vp, ctypes.POINTER(i32), i32, ctypes.POINTER(Group), i32,
        ctypes.POINTER(Member), i32, ctypes.POINTER(i64),
        ctypes.POINTER(i32), ctypes.POINTER(i32)]
    L.gemel_infer.argtypes = [vp, ctypes.POINTER(i32), i32,
                              ctypes.POINTER(vp), ctypes.POINTER(i32),
                              ctypes.POINTER(vp), vp]
    L.gemel_infer_noalloc.argtypes = L.gemel_infer.argtypes
    L.gemel_set_next_round.argtypes = [vp, ctypes.POINTER(i32), i32]
    L.gemel_load_order.argtypes = [vp, ctypes.POINTER(i32), i32,
                                   ctypes.POINTER(i32)]
    f64p = ctypes.POINTER(ctypes.c_double)
    L.gemel_sla_batches.argtypes = [i32, i32, f64p, f64p, i32,
                                    ctypes.c_double, ctypes.c_double,
                                    ctypes.POINTER(i32), f64p, f64p]
    L.gemel_profile_batches.argtypes = [vp, ctypes.POINTER(i32), i32, i32,
                                        i32, vp, f64p]
    L.gemel_model_outputs.argtypes = [vp, i32, ctypes.POINTER(i32)]
    L.gemel_output_shape.argtypes = [vp, i32, i32, i32,
                                     ctypes.POINTER(i64)]
    L.gemel_query.argtypes = [vp, i32, ctypes.POINTER(i64)]
    L.gemel_set_option.argtypes = [vp, i32, i64]
    L.gemel_profile.argtypes = [vp, ctypes.POINTER(KernelStat),
                                ctypes.POINTER(i32)]
    L.gemel_last_error.argtypes = [vp]
    L.gemel_last_error.restype = ctypes.c_char_p
    L.gemel_destroy.argtypes = [vp]
    for name in EXPORTED:
        if name != "gemel_last_error":
            getattr(L, name).restype = ctypes.c_int32
    return L


def lib():
    """Load libgemel.so (raises if it has not been built).

    torch brings its own HIP runtime whose soname equals the system one; it
    is loaded first so that libgemel binds to the same runtime instance
    (two HIP runtimes in one process do not share the device)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with "
                "`python -m paper_2201_07705_amd.build` (no fallback exists)")
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        L = ctypes.CDLL(LIB_PATH)
        rts = _hip_runtimes()
        if len(rts) > 1:
            raise RuntimeError(f"two HIP runtimes are loaded: {sorted(rts)}")
        _configure(L)
        _lib = L
    return _lib


def _fptr(a):
    return None if a is None else a.ctypes.data_as(_fp)


def layer_descs(layers, params):
    """Marshal layer dicts + parameter dicts into a LayerDesc array. Returns
    (array, keepalive list of the float32 arrays it points into)."""
    arr = (LayerDesc * len(layers))()
    keep = []
    for i, (l, p) in enumerate(zip(layers, params)):
        d = arr[i]
        d.op = OP[l["op"]]
        d.src0, d.src1 = l["src0"], l.get("src1", -1)
        d.cin, d.cout = l["cin"], l["cout"]
        d.kh, d.kw = l.get("kh", 1), l.get("kw", 1)
        d.stride, d.pad = l.get("stride", 1), l.get("pad", 0)
        d.act = ACT[l.get("act", "none")]
        d.act_slope = LEAKY_SLOPE if l.get("act") == "leaky" else 0.0
        d.res_src = l.get("res", -1)
        d.res_mode = RES_MODE[l.get("res_mode", "add_act")]
        d.is_output = 1 if l.get("out") else 0
        if p is not None:
            w = np.ascontiguousarray(p["w"], np.float32)
            keep.append(w)
            d.weight = _fptr(w)
            if p.get("b") is not None:
                b = np.ascontiguousarray(p["b"], np.float32)
                keep.append(b)
                d.bias = _fptr(b)
            if p.get("bn") is not None:
                g, be, mu, var, eps = p["bn"]
                vs = [np.ascontiguousarray(v, np.float32)
                      for v in (g, be, mu, var)]
                keep.extend(vs)
                d.bn_gamma, d.bn_beta, d.bn_mean, d.bn_var = \
                    [_fptr(v) for v in vs]
                d.bn_eps = eps
    return arr, keep


def sla_batches(cost_ms, sla_ms, fps, swap_ms=None, pipelined=True,
                library=None):
    """Per-model batch sizes under a per-frame deadline from a cost table
    [model][batch - 1] (ms): returns (batches, min frames/s, cycle ms)."""
    L = library or lib()
    n, nb = len(cost_ms), len(cost_ms[0])
    flat = (ctypes.c_double * (n * nb))(*[c for row in cost_ms for c in row])
    sw = (ctypes.c_double * n)(*swap_ms) if swap_ms is not None else None
    b = (ctypes.c_int32 * n)()
    v, t = ctypes.c_double(), ctypes.c_double()
    st = L.gemel_sla_batches(n, nb, flat, sw, 1 if pipelined else 0,
                             float(sla_ms), float(fps), b, ctypes.byref(v),
                             ctypes.byref(t))
    if st != OK:
        raise GemelError(st, "gemel_sla_batches: " + STATUS_NAMES.get(st, "?"))
    return list(b), v.value, t.value


class Context:
    """One libgemel context on one device."""

    def __init__(self, device=0, dtype="bf16", budget=0, library=None):
        self._lib = library or lib()
        self._h = ctypes.c_void_p()
        st = self._lib.gemel_create(ctypes.byref(self._h), device,
                                BF16 if dtype == "bf16" else F32, budget)
        if st != OK:
            raise GemelError(st, self._lib.gemel_last_error(None).decode())
        self.dtype = dtype
        self.device = device
        self._in_shape = {}
        self._out_ops = {}

    # -- raw calls (status returned, message on failure) --
    def _check(self, st):
        if st != OK:
            raise GemelError(st, self._lib.gemel_last_error(self._h).decode())
        return st

    def register_model(self, layers, params, in_chw):
        arr, keep = layer_descs(layers, params)
        mid = ctypes.c_int32(-1)
        self._check(self._lib.gemel_register_model(
            self._h, arr, len(layers), in_chw[0], in_chw[1], in_chw[2],
            ctypes.byref(mid)))
        del keep
        self._in_shape[mid.value] = tuple(in_chw)
        self._out_ops[mid.value] = [l["op"] for l in layers if l.get("out")]
        return mid.value

    def merge(self, groups):
        """groups: list of lists of (model_id, layer_index); first = source."""
        n = len(groups)
        garr = (Group * max(n, 1))()
        keep = []
        for i, g in enumerate(groups):
            m = (Member * len(g))(*[Member(a, b) for a, b in g])
            keep.append(m)
            garr[i].n_members = len(g)
            garr[i].members = ctypes.cast(m, ctypes.POINTER(Member))
        self._check(self._lib.gemel_merge(self._h, garr, n))

    def enumerate_groups(self, model_ids):
        """Candidate groups of the models (Section 5.3): a list of
        (total_bytes, [(model_id, layer_index), ...]) in descending order of
        memory, each accepted by merge() as it is."""
        n = len(model_ids)
        ids = (ctypes.c_int32 * max(n, 1))(*model_ids)
        ng, nm = ctypes.c_int32(), ctypes.c_int32()
        self._check(self._lib.gemel_enumerate_groups(
            self._h, ids, n, None, 0, None, 0, None, ctypes.byref(ng),
            ctypes.byref(nm)))
        garr = (Group * max(ng.value, 1))()
        marr = (Member * max(nm.value, 1))()
        nbytes = (ctypes.c_int64 * max(ng.value, 1))()
        self._check(self._lib.gemel_enumerate_groups(
            self._h, ids, n, garr, ng.value, marr, nm.value, nbytes,
            ctypes.byref(ng), ctypes.byref(nm)))
        out, at = [], 0
        for g in range(ng.value):
            k = garr[g].n_members
            out.append((nbytes[g], [(marr[at + j].model_id, marr[at + j].layer)
                                    for j in range(k)]))
            at += k
        return out

    def n_outputs(self, model_id):
        n = ctypes.c_int32()
        self._check(self._lib.gemel_model_outputs(self._h, model_id,
                                              ctypes.byref(n)))
        return n.value

    def output_shape(self, model_id, idx, n_frames):
        dims = (ctypes.c_int64 * 4)()
        self._check(self._lib.gemel_output_shape(self._h, model_id, idx,
                                             n_frames, dims))
        if self._out_ops.get(model_id, [None] * (idx + 1))[idx] == "fc":
            return (n_frames, dims[1])
        return (n_frames, dims[1], dims[2], dims[3])

    def query(self, key):
        v = ctypes.c_int64()
        self._check(self._lib.gemel_query(self._h, key, ctypes.byref(v)))
        return v.value

    def set_option(self, key, value):
        self._check(self._lib.gemel_set_option(self._h, key, value))

    def profile(self):
        """Per-round kernel statistics by family: {name: dict(launches,
        flops, bytes, ms)} and the number of profiled rounds."""
        st = (KernelStat * len(KERNEL_FAMILIES))()
        rounds = ctypes.c_int32()
        self._check(self._lib.gemel_profile(self._h, st, ctypes.byref(rounds)))
        return {name: dict(launches=s.launches, flops=s.flops, bytes=s.bytes,
                           ms=s.ms)
                for name, s in zip(KERNEL_FAMILIES, st)}, rounds.value

    def infer_raw(self, model_ids, frame_ptrs, n_frames, out_ptrs, stream,
                  noalloc=False):
        n = len(model_ids)
        ids = (ctypes.c_int32 * n)(*model_ids)
        fp = (ctypes.c_void_p * n)(*frame_ptrs)
        nf = (ctypes.c_int32 * n)(*n_frames)
        op = (ctypes.c_void_p * max(len(out_ptrs), 1))(*out_ptrs)
        fn = self._lib.gemel_infer_noalloc if noalloc else self._lib.gemel_infer
        return fn(self._h, ids, n, fp, nf, op, ctypes.c_void_p(stream))

    def set_next_round(self, model_ids):
        """Models of the round after the next infer (weight cache pins)."""
        n = len(model_ids)
        ids = (ctypes.c_int32 * max(n, 1))(*model_ids)
        self._check(self._lib.gemel_set_next_round(self._h, ids, n))

    def load_order(self, model_ids):
        """Sharing-aware round-robin load order of the models."""
        n = len(model_ids)
        ids = (ctypes.c_int32 * n)(*model_ids)
        out = (ctypes.c_int32 * n)()
        self._check(self._lib.gemel_load_order(self._h, ids, n, out))
        return list(out)

    def profile_batches(self, model_ids, max_batch, reps=5, stream=None):
        """Measured cost table [model][batch - 1] in ms (nondecreasing
        rows) of each model alone on 1..max_batch frames."""
        import torch
        n = len(model_ids)
        ids = (ctypes.c_int32 * n)(*model_ids)
        out = (ctypes.c_double * (n * max_batch))()
        s = stream if stream is not None else torch.cuda.current_stream()
        self._check(self._lib.gemel_profile_batches(
            self._h, ids, n, max_batch, reps, s.cuda_stream, out))
        return [list(out[i * max_batch:(i + 1) * max_batch])
                for i in range(n)]

    def close(self):
        if self._h:
            st = self._lib.gemel_destroy(self._h)
            self._h = ctypes.c_void_p()
            if st != OK:
                raise GemelError(st, "destroy found a device fault")

    def __del__(self):
        try:
            if self._h:
                self._lib.gemel_destroy(self._h)
        except Exception:
            pass

    # -- torch conveniences --
    def alloc_outputs(self, model_ids, n_frames, device="cuda"):
        import torch
        outs = []
        for mid, n in zip(model_ids, n_frames):
            outs.append([torch.empty(self.output_shape(mid, i, n),
                                     dtype=torch.float32, device=device)
                         for i in range(self.n_outputs(mid))])
        return outs

    def infer(self, model_ids, frames, stream=None, outputs=None,
              noalloc=False):
        """frames: list of float32 NCHW cuda tensors, one per model id.
        Returns (and fills) per-model lists of float32 output tensors.
        noalloc: call gemel_infer_noalloc (outputs must be given)."""
        import torch
        n_frames = [int(f.shape[0]) for f in frames]
        for f in frames:
            assert f.dtype == torch.float32 and f.is_cuda and \
                f.is_contiguous()
        if outputs is None:
            outputs = self.alloc_outputs(model_ids, n_frames,
                                         frames[0].device)
        out_ptrs = [t.data_ptr() for o in outputs for t in o]
        s = stream if stream is not None else torch.cuda.current_stream()
        self._check(self.infer_raw(model_ids, [f.data_ptr() for f in frames],
                                   n_frames, out_ptrs, s.cuda_stream,
                                   noalloc=noalloc))
        return outputs
