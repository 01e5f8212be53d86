"""Seeded synthetic inputs: weights, batch-norm statistics, biases, frames.

Serves both the HIP path and the oracle; holds none of the method's
arithmetic. Every draw comes from
``numpy.random.Generator(PCG64(SeedSequence([workload, model, stream])))``
with stream 0 = conv/fc weights, 1 = bias and batch-norm parameters,
2 = frames.

Distributions (the paper's trained weights and videos are not available,
so these stand in for them):
  weights   He-normal, std = sqrt(2 / fan_in), fan_in = cin*kh*kw
  BN        gamma ~ U(0.5, 1.5), beta ~ N(0, 0.1), mean 0, var 1, eps 1e-5
  bias      N(0, 0.1)
  frames    U[0, 1] or N(0, 1)
For bf16 workloads every value is snapped to the nearest bf16 (round to
nearest even) before either side sees it, so both sides start from
identical bytes.
"""

from __future__ import annotations

import numpy as np

STREAM_WEIGHTS, STREAM_AFFINE, STREAM_FRAMES = 0, 1, 2
BN_EPS = 1e-5


def rng(workload, model, stream):
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([int(workload), int(model), int(stream)])))


def snap_bf16(a):
    """Nearest bf16 value (ties to even) of each float32 element, returned
    as float32. Used to make generated inputs bf16-representable."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    out = u.astype(np.uint32).view(np.float32)
    nan = np.isnan(a)
    if nan.any():
        out = out.copy()
        out[nan] = np.nan
    return out


def model_params(layers, workload, model, bf16):
    """Per-layer parameter dicts (None for layers without parameters).

    conv weight is OIHW [cout][cin][kh][kw]; fc weight is [cout][cin] with
    the input flattened in NCHW order. 'bn' is (gamma, beta, mean, var, eps).
    """
    gw = rng(workload, model, STREAM_WEIGHTS)
    ga = rng(workload, model, STREAM_AFFINE)
    snap = snap_bf16 if bf16 else (lambda a: a)
    out = []
    for l in layers:
        if l["op"] not in ("conv", "fc"):
            out.append(None)
            continue
        if l["op"] == "conv":
            shape = (l["cout"], l["cin"], l["kh"], l["kw"])
        else:
            shape = (l["cout"], l["cin"])
        fan_in = int(np.prod(shape[1:]))
        w = gw.standard_normal(shape, dtype=np.float32)
        w *= np.float32(np.sqrt(2.0 / fan_in))
        p = {"w": snap(w), "b": None, "bn": None}
        if l["bias"]:
            p["b"] = (0.1 * ga.standard_normal(l["cout"])).astype(np.float32)
        if l["bn"]:
            gamma = ga.uniform(0.5, 1.5, l["cout"]).astype(np.float32)
            beta = (0.1 * ga.standard_normal(l["cout"])).astype(np.float32)
            p["bn"] = (gamma, beta, np.zeros(l["cout"], np.float32),
                       np.ones(l["cout"], np.float32), BN_EPS)
        out.append(p)
    return out


def frames(workload, model, n, chw, dist, bf16):
    """n frames of shape chw, NCHW float32."""
    g = rng(workload, model, STREAM_FRAMES)
    shape = (n,) + tuple(chw)
    if dist == "uniform":
        f = g.random(shape, dtype=np.float32)
    elif dist == "normal":
        f = g.standard_normal(shape, dtype=np.float32)
    else:
        raise ValueError(dist)
    return snap_bf16(f) if bf16 else f
