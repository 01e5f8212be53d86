"""Shared helpers of the GPU tests: run a workload through the C ABI of
libgemel and compare with the oracle on the same seeded inputs."""

from __future__ import annotations

import sys
import time

import numpy as np

BF16_TOL = 2e-2      # normwise max relative error for bf16 workloads
F32_TOL = 1e-4       # the same for float32 workloads

# One record per compared output (tag, model, output, normwise error, argmax
# vectors compared, near-tie exemptions, mismatches); printed at the end of
# the session by tests/conftest.py.
PARITY = []


def log(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)
    sys.stdout.flush()


def normwise(got, ref):
    """max |g - r| / max |r| over one output tensor."""
    den = float(np.max(np.abs(ref)))
    if den == 0.0:
        return float(np.max(np.abs(got)))
    return float(np.max(np.abs(got.astype(np.float64) - ref)) / den)


def argmax_check(got, ref):
    """Per frame, the arg-max class must agree unless the oracle's top-2 gap
    is within twice the frame's max abs error (a near tie that bf16 storage
    may legitimately flip). Returns (mismatches, near_ties)."""
    g = got.reshape(got.shape[0], -1)
    r = ref.reshape(ref.shape[0], -1)
    bad, ties = 0, 0
    for i in range(g.shape[0]):
        err = float(np.max(np.abs(g[i] - r[i])))
        top2 = np.sort(r[i])[-2:]
        margin = float(top2[1] - top2[0])
        if np.argmax(g[i]) != np.argmax(r[i]):
            if margin > 2 * err:
                bad += 1
            else:
                ties += 1
    return bad, ties


def yolo_class_vectors(t, classes=80):
    """Class scores per (anchor, cell) of a [n, 3*(5+classes), S, S] map, as
    rows of a [n*3*S*S, classes] array."""
    n, c, h, w = t.shape
    a = t.reshape(n, 3, 5 + classes, h, w)[:, :, 5:]
    return np.ascontiguousarray(a.transpose(0, 1, 3, 4, 2)).reshape(-1, classes)


class GpuWorkload:
    """A workload registered and merged in one libgemel context."""

    def __init__(self, wl, params=None, budget=0, device=0, merge=True):
        import paper_2201_07705_amd as P
        self.wl = wl
        self.ctx = P.Context(device, wl.dtype,
                             budget if isinstance(budget, int) else 0)
        self.params = params or [wl.params(i) for i in range(len(wl.models))]
        self.ids = [self.ctx.register_model(m.layers, self.params[i],
                                            m.in_chw)
                    for i, m in enumerate(wl.models)]
        if merge:
            self.ctx.merge([[(self.ids[a], b) for a, b in g]
                            for g in wl.groups])
        from paper_2201_07705_amd import gemel as G
        for name, value in wl.options.items():
            self.ctx.set_option(getattr(G, "OPT_" + name.upper()), int(value))
        if budget == "auto" and wl.budget_frac:
            from paper_2201_07705_amd import gemel as G
            unmerged = self.ctx.query(G.Q_UNMERGED_BYTES)
            self.ctx.set_option(G.OPT_WEIGHT_BUDGET,
                                int(wl.budget_frac * unmerged))

    def run(self, frames, stream=None, order=None, repeat=1):
        import torch
        order = list(range(len(self.ids))) if order is None else order
        dev = [torch.from_numpy(np.ascontiguousarray(frames[i])).cuda()
               for i in order]
        s = stream or torch.cuda.Stream()
        outs = None
        with torch.cuda.stream(s):
            for _ in range(repeat):
                outs = self.ctx.infer([self.ids[i] for i in order], dev,
                                      stream=s, outputs=outs)
        s.synchronize()
        res = [None] * len(self.ids)
        for k, i in enumerate(order):
            res[i] = [o.cpu().numpy() for o in outs[k]]
        return res

    def close(self):
        self.ctx.close()


def oracle_outputs(wl, params, frames, round_act=False):
    from oracle import model as om
    return om.run_workload(wl.models, params, frames, wl.groups, round_act)


def compare(wl, got, ref, tol=None, check_argmax=True, check_norm=True,
            tag=""):
    """Assert normwise error per output and arg-max agreement (classifier
    logits per frame; YOLO class scores per anchor and cell). Every output
    is checked and recorded before the first failure is raised."""
    tol = tol or (BF16_TOL if wl.bf16 else F32_TOL)
    worst = 0.0
    errors = []
    for mi, (g_outs, r_outs) in enumerate(zip(got, ref)):
        assert len(g_outs) == len(r_outs)
        for oi, (g, r) in enumerate(zip(g_outs, r_outs)):
            assert g.shape == r.shape, (tag, mi, oi, g.shape, r.shape)
            assert np.all(np.isfinite(g)), (tag, mi, oi)
            e = normwise(g, r)
            worst = max(worst, e)
            rec = {"tag": tag, "model": mi, "output": oi, "normwise": e,
                   "vectors": 0, "near_ties": 0, "mismatches": 0}
            if check_norm and e > tol:
                errors.append(f"{tag} model {mi} output {oi}: normwise "
                              f"error {e:.3e} > {tol:.0e}")
            vec = None
            if check_argmax and g.ndim == 2:
                vec = (g, r)
            if check_argmax and g.ndim == 4 and g.shape[1] == 255:
                vec = (yolo_class_vectors(g), yolo_class_vectors(r))
            if vec is not None:
                bad, ties = argmax_check(*vec)
                rec.update(vectors=int(vec[0].shape[0]), near_ties=ties,
                           mismatches=bad)
                if bad:
                    errors.append(f"{tag} model {mi} output {oi}: {bad} "
                                  "argmax mismatches beyond near ties")
            PARITY.append(rec)
            log(f"{tag} model {mi} output {oi}: normwise {e:.3e}"
                + (f", argmax over {rec['vectors']} vectors, "
                   f"{rec['near_ties']} near-tie exemptions, "
                   f"{rec['mismatches']} mismatches"
                   if rec["vectors"] else ""))
    assert not errors, "; ".join(errors)
    return worst
