"""Oracle model evaluation: walk one model's layer graph on its own frames.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What merging means (Section 4 of the paper): architecturally identical
layers are shared so that a single copy of each shared layer's definition
and weights serves every model that contains it; layer outputs are never
shared, because models may look at different videos. Hence the merged
result of a model is that model evaluated alone with its *effective*
weights: a merged layer holds the weights of its group's source member
(Section 5.3 seeds a merged group from one member's weights; here the source
is the group's first member). ``effective_params`` builds those weights and
``run_model`` evaluates one model; nothing here batches models together.

Step definitions (plain textbook definitions; the paper relies on them
without restating them):
  conv       oracle.conv2d (cross-correlation, zero padding)
  batch norm y = gamma * (z - mean) / sqrt(var + eps) + beta (unfolded)
  relu       max(0, y);  leaky  y if y > 0 else 0.1 * y
  residual   'add_act': act(z + r) (ResNet);  'act_add': act(z) + r (Darknet)
  maxpool    max over the window, padding taken as -inf
  avgpool    global mean over H x W
  upsample   nearest neighbour, y[.., h, w] = x[.., h // 2, w // 2]
  concat     along channels, [src0, src1]
  fc         input flattened in NCHW order, oracle.fc
"""

from __future__ import annotations

import numpy as np

from . import conv2d, fc

LEAKY_SLOPE = 0.1


def effective_params(params, groups):
    """Per-model parameter lists after merging: every member of a group uses
    the parameters (weights, bias and batch-norm) of the group's first
    member. ``params`` is a list (one per model) of per-layer dicts."""
    eff = [list(p) for p in params]
    for g in groups:
        sm, sl = g[0]
        for (m, l) in g[1:]:
            eff[m][l] = params[sm][sl]
    return eff


def round_bf16(a):
    """Round float32 values to the nearest bfloat16 (ties to even); used only
    by the diagnostic mode that stores activations in bf16."""
    a = np.ascontiguousarray(a, np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).reshape(a.shape)


def _act(y, act):
    if act == "relu":
        return np.maximum(y, np.float32(0))
    if act == "leaky":
        return np.where(y > 0, y, (np.float64(LEAKY_SLOPE) * y)
                        .astype(np.float32))
    assert act == "none", act
    return y


def _bn(z, bn):
    gamma, beta, mean, var, eps = bn
    g = gamma.astype(np.float64)[None, :, None, None]
    b = beta.astype(np.float64)[None, :, None, None]
    m = mean.astype(np.float64)[None, :, None, None]
    v = var.astype(np.float64)[None, :, None, None]
    return (g * (z.astype(np.float64) - m) / np.sqrt(v + eps) + b) \
        .astype(np.float32)


def _maxpool(x, k, s, p):
    n, c, h, w = x.shape
    ho = (h + 2 * p - k) // s + 1
    wo = (w + 2 * p - k) // s + 1
    xp = np.full((n, c, h + 2 * p, w + 2 * p), -np.inf, np.float32)
    xp[:, :, p:p + h, p:p + w] = x
    y = np.full((n, c, ho, wo), -np.inf, np.float32)
    for i in range(k):
        for j in range(k):
            y = np.maximum(y, xp[:, :, i:i + s * (ho - 1) + 1:s,
                                 j:j + s * (wo - 1) + 1:s])
    return y


def _avgpool(x):
    return x.astype(np.float64).mean(axis=(2, 3), keepdims=True) \
        .astype(np.float32)


def _upsample2x(x):
    return x.repeat(2, axis=2).repeat(2, axis=3)


def run_model(layers, params, frames, round_act=False):
    """Evaluate one model. ``frames`` is NCHW float32; returns the outputs of
    the layers marked ``out`` in layer order (conv outputs NCHW, fc outputs
    [n, classes]). ``round_act`` stores every layer output in bf16 (a
    diagnostic that separates precision drift from kernel errors)."""
    x0 = np.ascontiguousarray(frames, np.float32)
    vals = [None] * len(layers)
    outs = []
    for i, l in enumerate(layers):
        src = x0 if l["src0"] < 0 else vals[l["src0"]]
        op = l["op"]
        p = params[i]
        if op == "conv":
            z = conv2d(src, p["w"], p["b"], l["stride"], l["pad"])
            if p["bn"] is not None:
                z = _bn(z, p["bn"])
        elif op == "fc":
            z = fc(src.reshape(src.shape[0], -1), p["w"], p["b"])
        elif op == "maxpool":
            z = _maxpool(src, l["kh"], l["stride"], l["pad"])
        elif op == "avgpool":
            z = _avgpool(src)
        elif op == "upsample":
            z = _upsample2x(src)
        elif op == "concat":
            z = np.concatenate([src, vals[l["src1"]]], axis=1)
        else:
            raise ValueError(op)
        if op in ("conv", "fc"):
            if l["res"] >= 0:
                r = vals[l["res"]]
                if l["res_mode"] == "add_act":
                    z = _act(z + r, l["act"])
                else:
                    z = _act(z, l["act"]) + r
            else:
                z = _act(z, l["act"])
        if round_act and not l["out"]:
            z = round_bf16(z)
        vals[i] = z
        if l["out"]:
            outs.append(z.reshape(z.shape[0], -1) if op == "fc" else z)
    return outs


def run_workload(models, params, frames, groups, round_act=False):
    """Outputs of every model of a merged workload: per model, the model run
    alone on its frames with its effective (post-merge) parameters."""
    eff = effective_params(params, groups)
    return [run_model(m.layers, eff[i], frames[i], round_act)
            for i, m in enumerate(models)]
