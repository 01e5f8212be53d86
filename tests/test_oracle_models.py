"""Model-level pins of the oracle.

Each architecture is written out again below as a textbook forward pass in
torch float64 (torch.nn.functional conv2d / batch_norm / max_pool2d /
interpolate / linear), reading the same seeded parameters by layer name.
This pins the oracle's graph walk, its primitives and the architecture
descriptors together against an independent formulation. The merging
invariants (Section 4: one copy of a shared layer serves every model that
includes it; intermediates are not shared) are pinned on the oracle itself.
"""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import model as om
from workloads import configs, gen, zoo


def _t(a):
    return torch.from_numpy(np.asarray(a)).double()


def _by_name(layers, params):
    """Seeded parameters keyed by layer name, as float64 torch tensors."""
    d = {}
    for l, p in zip(layers, params):
        if p is None:
            continue
        bn = None
        if p["bn"] is not None:
            g, b, m, v, eps = p["bn"]
            bn = (_t(g), _t(b), _t(m), _t(v), eps)
        d[l["name"]] = {"w": _t(p["w"]),
                        "b": None if p["b"] is None else _t(p["b"]),
                        "bn": bn}
    return d


def _conv(P, name, x, stride, pad, act=None):
    p = P[name]
    y = F.conv2d(x, p["w"], p["b"], stride=stride, padding=pad)
    if p["bn"] is not None:
        g, b, m, v, eps = p["bn"]
        y = F.batch_norm(y, m, v, g, b, False, 0.0, eps)
    if act == "relu":
        y = F.relu(y)
    elif act == "leaky":
        y = F.leaky_relu(y, 0.1)
    return y


def torch_resnet(P, x, depth):
    kind, counts = {18: ("basic", [2, 2, 2, 2]),
                    50: ("bottleneck", [3, 4, 6, 3])}[depth]
    x = _conv(P, "conv1", x, 2, 3, "relu")
    x = F.max_pool2d(x, 3, 2, 1)
    for si, n in enumerate(counts):
        for bi in range(n):
            s = 2 if (bi == 0 and si > 0) else 1
            p = f"layer{si + 1}.{bi}"
            short = _conv(P, p + ".downsample", x, s, 0) \
                if p + ".downsample" in P else x
            if kind == "basic":
                y = _conv(P, p + ".conv1", x, s, 1, "relu")
                y = _conv(P, p + ".conv2", y, 1, 1)
            else:
                y = _conv(P, p + ".conv1", x, 1, 0, "relu")
                y = _conv(P, p + ".conv2", y, s, 1, "relu")
                y = _conv(P, p + ".conv3", y, 1, 0)
            x = F.relu(y + short)
    x = x.mean(dim=(2, 3))
    return [F.linear(x, P["fc"]["w"], P["fc"]["b"])]


def torch_vgg(P, x):
    ci = pi = 0
    for v in zoo._VGG_CFG[16]:
        if v == "M":
            x = F.max_pool2d(x, 2, 2)
            pi += 1
        else:
            x = _conv(P, f"features.conv{ci}", x, 1, 1, "relu")
            ci += 1
    x = torch.flatten(x, 1)
    x = F.relu(F.linear(x, P["classifier.fc6"]["w"], P["classifier.fc6"]["b"]))
    x = F.relu(F.linear(x, P["classifier.fc7"]["w"], P["classifier.fc7"]["b"]))
    return [F.linear(x, P["classifier.fc8"]["w"], P["classifier.fc8"]["b"])]


def torch_yolov3(P, x):
    x = _conv(P, "backbone.conv0", x, 1, 1, "leaky")
    taps = []
    for si, n in enumerate([1, 2, 8, 8, 4]):
        x = _conv(P, f"backbone.down{si}", x, 2, 1, "leaky")
        for bi in range(n):
            p = f"backbone.stage{si}.{bi}"
            y = _conv(P, p + ".conv1", x, 1, 0, "leaky")
            x = x + _conv(P, p + ".conv2", y, 1, 1, "leaky")
        taps.append(x)
    outs = []
    for hi, tap in enumerate([None, taps[3], taps[2]]):
        p = f"head{hi}"
        if tap is not None:
            r = _conv(P, p + ".route", route, 1, 0, "leaky")
            x = torch.cat([F.interpolate(r, scale_factor=2, mode="nearest"),
                           tap], dim=1)
        for j in range(5):
            k = 1 if j % 2 == 0 else 3
            x = _conv(P, f"{p}.conv{j}", x, 1, k // 2, "leaky")
        route = x
        y = _conv(P, p + ".conv5", x, 1, 1, "leaky")
        outs.append(_conv(P, p + ".out", y, 1, 0))
    return outs


def normwise(a, b):
    return float(np.max(np.abs(a - b)) / np.max(np.abs(b)))


@pytest.mark.parametrize("arch,res,fn", [
    ("resnet18", 64, lambda P, x: torch_resnet(P, x, 18)),
    ("resnet50", 64, lambda P, x: torch_resnet(P, x, 50)),
    ("vgg16", 32, torch_vgg),
    ("yolov3", 64, torch_yolov3),
])
def test_oracle_matches_torch_float64_architecture(arch, res, fn):
    layers = zoo.vgg(16, 1000, res) if arch == "vgg16" else zoo.build(arch)
    params = gen.model_params(layers, 99, 0, bf16=True)
    x = gen.frames(99, 0, 2, (3, res, res), "normal", bf16=True)
    got = om.run_model(layers, params, x)
    ref = fn(_by_name(layers, params), torch.from_numpy(x).double())
    assert len(got) == len(ref)
    for g, r in zip(got, ref):
        r = r.numpy()
        assert g.shape == r.shape
        assert normwise(g, r) < 1e-5


def test_merged_equals_unmerged_with_identical_shared_weights():
    """When every member already holds the source's weights, merging must
    not change any model's output (bitwise, inside the oracle)."""
    w = configs.resnet18x2(res=32, frames=2)
    p0 = w.params(0)
    p1 = w.params(1)
    # give model 1 model 0's weights on every shared layer
    for g in w.groups:
        (m0, l0), (m1, l1) = g
        p1[l1] = p0[l0]
    fr = [w.frames(0), w.frames(1)]
    merged = om.run_workload(w.models, [p0, p1], fr, w.groups)
    unmerged = [om.run_model(w.models[i].layers, [p0, p1][i], fr[i])
                for i in range(2)]
    for a, b in zip(merged, unmerged):
        for x, y in zip(a, b):
            assert np.array_equal(x, y)


def test_effective_params_take_the_source_member():
    w = configs.resnet18x2(res=32, frames=1)
    ps = [w.params(0), w.params(1)]
    eff = om.effective_params(ps, w.groups)
    shared = {(m, l) for g in w.groups for (m, l) in g}
    for g in w.groups:
        (sm, sl) = g[0]
        for (m, l) in g:
            assert eff[m][l] is ps[sm][sl]
    # unshared layers (the two FC heads) keep their own weights
    for m in range(2):
        for l in range(len(w.models[m].layers)):
            if (m, l) not in shared:
                assert eff[m][l] is ps[m][l]
    # and the merged models really differ from the unmerged ones
    fr = [w.frames(0), w.frames(1)]
    a = om.run_workload(w.models, ps, fr, w.groups)[1][0]
    b = om.run_model(w.models[1].layers, ps[1], fr[1])[0]
    assert not np.array_equal(a, b)


def test_frame_permutation_permutes_outputs_bitwise():
    w = configs.tiny2(res=16, frames=5)
    p = w.params(0)
    x = w.frames(0)
    perm = [3, 0, 4, 2, 1]
    a = om.run_model(w.models[0].layers, p, x)[0]
    b = om.run_model(w.models[0].layers, p, x[perm])[0]
    assert np.array_equal(a[perm], b)


def test_diagnostic_bf16_storage_stays_close():
    w = configs.resnet18x2(res=32, frames=2)
    p = w.params(0)
    x = w.frames(0)
    a = om.run_model(w.models[0].layers, p, x)[0]
    b = om.run_model(w.models[0].layers, p, x, round_act=True)[0]
    e = normwise(b, a)
    assert 0 < e < 2e-2
