"""Pins of the architecture descriptors and workload definitions against
facts printed in the paper (tests/golden/paper_memory_facts.txt) and the
published parameter and operation counts of the standard architectures."""

import os

import numpy as np
import pytest

from workloads import configs, gen, zoo

GOLDEN = os.path.join(os.path.dirname(__file__), "golden",
                      "paper_memory_facts.txt")


def _facts(kind):
    out = []
    for line in open(GOLDEN):
        line = line.split("#")[0].split()
        if line and line[0] == kind:
            out.append(line[1:])
    return out


@pytest.mark.parametrize("arch,gb", _facts("table1"))
def test_table1_load_memory_within_rounding(arch, gb):
    # fp32 parameters in decimal GB against Table 1's two-decimal figures;
    # the paper does not state its counting convention, so allow +-0.02 GB
    bytes_fp32 = 4 * zoo.param_count(zoo.build(arch))
    assert abs(bytes_fp32 / 1e9 - float(gb)) <= 0.02


def test_vgg16_fc6_is_392_mib():
    (arch, name, mib), = _facts("fc6_mib")
    layers = zoo.build(arch)
    l = next(l for l in layers if l["name"] == name)
    assert l["cin"] == 512 * 7 * 7 and l["cout"] == 4096
    b = 4 * zoo.layer_param_count(l)
    assert round(b / 2 ** 20) == int(mib)


@pytest.mark.parametrize("arch,params", [
    ("resnet18", 11_689_512), ("resnet34", 21_797_672),
    ("resnet50", 25_557_032), ("resnet152", 60_192_808),
    ("vgg16", 138_357_544), ("vgg19", 143_667_240),
    ("yolov3", 61_949_149),
])
def test_published_parameter_totals(arch, params):
    assert zoo.param_count(zoo.build(arch)) == params


def test_yolov3_416_operation_count():
    # the Darknet reference implementation reports 65.864 BFLOPs at 416x416
    f = 2 * zoo.macs(zoo.yolov3(), (3, 416, 416))
    assert abs(f / 1e9 - 65.864) < 0.001


@pytest.mark.parametrize("arch,convs", [("resnet18", 20), ("resnet34", 36),
                                        ("resnet50", 53), ("yolov3", 75),
                                        ("vgg16", 13), ("vgg19", 16)])
def test_conv_counts(arch, convs):
    assert sum(l["op"] == "conv" for l in zoo.build(arch)) == convs


def test_topological_order_and_shapes():
    for arch in ("resnet18", "resnet152", "vgg19", "yolov3"):
        layers = zoo.build(arch)
        for i, l in enumerate(layers):
            assert l["src0"] < i and l["src1"] < i and l["res"] < i
        sh = zoo.shapes(layers, (3, 416, 416) if arch == "yolov3"
                        else (3, 224, 224))
        for i, l in enumerate(layers):
            if l["res"] >= 0:
                assert sh[l["res"]] == sh[i]
            if l["op"] == "fc":
                c, h, w = sh[l["src0"]] if l["src0"] >= 0 else (3, 224, 224)
                assert c * h * w == l["cin"]
    outs = [s for l, s in zip(zoo.yolov3(), zoo.shapes(zoo.yolov3(),
                                                       (3, 416, 416)))
            if l["out"]]
    assert outs == [(255, 13, 13), (255, 26, 26), (255, 52, 52)]


def test_workload_flops_match_config_sizes():
    expect = {"tiny2": 0.0159, "resnet18x2": 29.02, "r50x2_vgg16x2": 625.8,
              "yolov3x3": 790.4, "mix8_budget40": 1507.1}
    for name, gf in expect.items():
        w = configs.get(name)
        assert abs(w.flops() / 1e9 - gf) / gf < 2e-3, name


def test_groups_are_architecturally_identical_and_disjoint():
    keys = ("op", "cin", "cout", "kh", "kw", "stride", "pad", "bias", "bn",
            "act", "res_mode")
    for name in configs.WORKLOADS:
        w = configs.get(name)
        seen = set()
        for g in w.groups:
            assert len(g) >= 2
            src = w.models[g[0][0]].layers[g[0][1]]
            for (m, l) in g:
                assert (m, l) not in seen
                seen.add((m, l))
                lay = w.models[m].layers[l]
                assert all(lay[k] == src[k] for k in keys), (name, lay["name"])


def test_generators_are_seeded_and_bf16_representable():
    w = configs.resnet18x2(res=32, frames=2)
    a, b = w.params(0), w.params(0)
    assert all(np.array_equal(x["w"], y["w"]) for x, y in zip(a, b) if x)
    c = w.params(1)
    assert not np.array_equal(a[0]["w"], c[0]["w"])
    f = w.frames(0)
    for arr in (f, a[0]["w"]):
        assert np.all((arr.view(np.uint32) & 0xFFFF) == 0)
    # He-normal fan_in scale on a large layer
    std = a[-1]["w"].std()
    assert abs(std / np.sqrt(2 / 512) - 1) < 0.05


def test_snap_bf16_round_to_nearest_even():
    v = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 3.0],
                 np.float32)
    np.testing.assert_array_equal(gen.snap_bf16(v),
                                  [1.0, 1 + 2 ** -6, -1.0, 3.0])
