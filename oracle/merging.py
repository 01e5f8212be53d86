"""Oracle of the merging heuristic's first step: candidate groups of a workload.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Section 5.3 of the paper: the heuristic starts by listing every layer that
appears in the workload, noting which models it appears in and where, and
the total memory all its appearances consume; all appearances of one layer
form a group. The list is sorted by that total memory, largest first (a
100 MB layer in four models comes before a 120 MB layer in three), so that
the groups whose merging saves the most are tried first. Section 4.1: a
layer can be shared only where it is architecturally identical, i.e. of
the same type with the same type-specific properties; the weights may
differ.

Readings taken here:
  - only layers with parameters (conv, fc) are listed: a layer without
    weights has nothing to share, and batch norm is part of its conv;
  - identity: type, input and output channels, kernel size, stride and
    padding, bias and batch-norm presence, and for an fc the (C, H, W) of
    the tensor it flattens (its weight columns follow that order);
  - the memory of one appearance is its parameter count (weights, cout for
    a bias, 4 * cout for batch norm: gamma, beta, mean, variance) times the
    element size; a group's memory is the sum over its appearances;
  - only groups with two or more appearances are candidates; ties in memory
    keep the order of first appearance; within a group, appearances are in
    model order, then layer order, and the first is the weight source.
"""

from __future__ import annotations


def output_shapes(layers, in_chw):
    """(C, H, W) of every layer's output, from the layer definitions."""
    out = []
    for l in layers:
        c, h, w = in_chw if l["src0"] < 0 else out[l["src0"]]
        op = l["op"]
        if op in ("conv", "maxpool"):
            out.append((l["cout"],
                        (h + 2 * l["pad"] - l["kh"]) // l["stride"] + 1,
                        (w + 2 * l["pad"] - l["kw"]) // l["stride"] + 1))
        elif op == "avgpool":
            out.append((c, 1, 1))
        elif op == "fc":
            out.append((l["cout"], 1, 1))
        elif op == "upsample":
            out.append((c, 2 * h, 2 * w))
        elif op == "concat":
            out.append((c + out[l["src1"]][0], h, w))
        else:
            raise ValueError(op)
    return out


def identity(layers, shapes, in_chw, i):
    """Architectural identity of layer i (None for a layer without
    parameters)."""
    l = layers[i]
    if l["op"] not in ("conv", "fc"):
        return None
    producer = (0, 0, 0)
    if l["op"] == "fc":
        producer = in_chw if l["src0"] < 0 else shapes[l["src0"]]
    return (l["op"], l["cin"], l["cout"], l.get("kh", 1), l.get("kw", 1),
            l.get("stride", 1), l.get("pad", 0), bool(l.get("bias")),
            bool(l.get("bn"))) + tuple(producer)


def param_count(l):
    """Parameters of one conv or fc layer."""
    k = l.get("kh", 1) * l.get("kw", 1) if l["op"] == "conv" else 1
    n = l["cout"] * l["cin"] * k
    if l.get("bias"):
        n += l["cout"]
    if l.get("bn"):
        n += 4 * l["cout"]
    return n


def candidate_groups(models, elem_bytes):
    """models: list of (model_id, layers, in_chw). Returns the candidate
    groups, most memory first: [(total_bytes, [(model_id, layer), ...])]."""
    groups = {}     # identity -> [total bytes, members, first position]
    for pos, (mid, layers, in_chw) in enumerate(models):
        shapes = output_shapes(layers, in_chw)
        for i in range(len(layers)):
            key = identity(layers, shapes, in_chw, i)
            if key is None:
                continue
            g = groups.setdefault(key, [0, [], (pos, i)])
            g[0] += param_count(layers[i]) * elem_bytes
            g[1].append((mid, i))
    cands = [g for g in groups.values() if len(g[1]) >= 2]
    cands.sort(key=lambda g: (-g[0], g[2]))
    return [(g[0], g[1]) for g in cands]


def shared_layer_count(models, count_bn_separately=False):
    """Layers two models can share (the figures of the paper's Appendix
    comparing model variants): for each identity, the smaller of its two
    appearance counts, summed. With count_bn_separately, a conv with batch
    norm counts as two layers (conv and batch norm), as the paper counts
    them."""
    (a_layers, a_in), (b_layers, b_in) = models
    counts = []
    for layers, in_chw in ((a_layers, a_in), (b_layers, b_in)):
        shapes = output_shapes(layers, in_chw)
        c = {}
        for i in range(len(layers)):
            key = identity(layers, shapes, in_chw, i)
            if key is None:
                continue
            w = 2 if count_bn_separately and layers[i].get("bn") else 1
            c[key] = c.get(key, 0) + w
        counts.append(c)
    return sum(min(n, counts[1].get(k, 0)) for k, n in counts[0].items())


def layer_count(layers, count_bn_separately=False):
    """Parametric layers of a model (batch norm separately if asked)."""
    return sum((2 if count_bn_separately and l.get("bn") else 1)
               for l in layers if l["op"] in ("conv", "fc"))
