"""The merged multi-model workloads: which models, how many frames each,
which layers are merged, data type and weight budget.

A workload's sharing map is a list of groups; a group lists
``(model_index, layer_index)`` appearances of one architecturally identical
layer, the first appearance being the one whose weights every member uses
(the paper seeds a merged layer with one member's weights, Section 5.3).

Full-size workloads (the paper's video frames are stood in for by seeded
synthetic frames of the same shape):
  tiny2          two tiny CNNs, fp32, 1 frame each, 3x32x32 U[0,1]
  resnet18x2     2x ResNet-18, bf16, 4 frames each, 3x224x224 N(0,1); every
                 conv stage merged, FC heads 512->1000 / 512->80 per model
  r50x2_vgg16x2  2x ResNet-50 sharing stem + layer1..3 (layer4 and FC heads
                 2048->1000 / 2048->20 per model) and 2x VGG-16 sharing all
                 13 convs (FC stacks per model, last FC ->1000 / ->10);
                 bf16, 8 frames each, 3x224x224 N(0,1)
  yolov3x3       3x YOLOv3 sharing the Darknet-53 backbone, heads per model;
                 bf16, 4 frames each, 3x416x416 U[0,1]
  mix8_budget40  ResNet-152 x2, ResNet-50 x3, VGG-19 x3; stem + layer1 shared
                 by all five ResNets, layer2 shared within each depth, VGG-19
                 conv blocks 1-3 shared; bf16, 8 frames each, 3x224x224 N(0,1);
                 resident weights capped at 40% of the unmerged weight bytes
"""

from __future__ import annotations

from dataclasses import dataclass, field

from . import gen, zoo


@dataclass
class ModelSpec:
    name: str
    arch: str
    layers: list
    n_frames: int
    in_chw: tuple


@dataclass
class Workload:
    name: str
    index: int                      # seed key of the workload
    dtype: str                      # 'f32' | 'bf16'
    models: list
    groups: list = field(default_factory=list)
    frame_dist: str = "normal"
    budget_frac: float = 0.0        # 0 = unlimited
    # library options the workload runs with (gemel_set_option names
    # without the OPT_ prefix), in the tests and the benchmark alike
    options: dict = field(default_factory=dict)

    @property
    def bf16(self):
        return self.dtype == "bf16"

    def params(self, mi):
        return gen.model_params(self.models[mi].layers, self.index, mi,
                                self.bf16)

    def frames(self, mi, n=None):
        m = self.models[mi]
        return gen.frames(self.index, mi, m.n_frames if n is None else n,
                          m.in_chw, self.frame_dist, self.bf16)

    def total_frames(self):
        return sum(m.n_frames for m in self.models)

    def flops(self):
        """2 * MAC over every executed conv and FC, all frames (merging does
        not change the arithmetic a model performs)."""
        return sum(2 * zoo.macs(m.layers, m.in_chw) * m.n_frames
                   for m in self.models)

    def merged_conv_flops(self):
        """FLOPs of conv layers that run in a merged (multi-model) group."""
        merged = set()
        for g in self.groups:
            if len(g) > 1:
                merged.update(g)
        tot = 0
        for mi, m in enumerate(self.models):
            sh = zoo.shapes(m.layers, m.in_chw)
            for li, l in enumerate(m.layers):
                if l["op"] == "conv" and (mi, li) in merged:
                    c, h, w = sh[li]
                    tot += 2 * c * h * w * l["cin"] * l["kh"] * l["kw"] \
                        * m.n_frames
        return tot


def share_by_name(models, model_idx, pred):
    """Groups for every layer name accepted by ``pred`` that appears in all
    of ``model_idx``; members ordered as model_idx (first = weight source)."""
    first = models[model_idx[0]].layers
    groups = []
    for li, l in enumerate(first):
        if not pred(l["name"]):
            continue
        g = []
        for mi in model_idx:
            names = [x["name"] for x in models[mi].layers]
            if l["name"] not in names:
                break
            g.append((mi, names.index(l["name"])))
        else:
            groups.append(g)
    return groups


def _resnet_prefix(stages):
    def pred(name):
        if name in ("conv1", "maxpool"):
            return True
        return any(name.startswith(f"layer{s}.") for s in stages)
    return pred


def tiny2(res=32, frames=1):
    chw = (3, res, res)
    models = [ModelSpec("tiny_a", "tiny", zoo.tiny(10), frames, chw),
              ModelSpec("tiny_b", "tiny", zoo.tiny(10), frames, chw)]
    groups = share_by_name(models, [0, 1], lambda n: n in ("conv1", "conv2"))
    return Workload("tiny2", 0, "f32", models, groups, "uniform")


def resnet18x2(res=224, frames=4):
    chw = (3, res, res)
    models = [ModelSpec("r18_a", "resnet18", zoo.resnet(18, 1000), frames, chw),
              ModelSpec("r18_b", "resnet18", zoo.resnet(18, 80), frames, chw)]
    groups = share_by_name(models, [0, 1], _resnet_prefix([1, 2, 3, 4]))
    groups += share_by_name(models, [0, 1], lambda n: n == "avgpool")
    return Workload("resnet18x2", 1, "bf16", models, groups, "normal")


def r50x2_vgg16x2(res=224, frames=8):
    chw = (3, res, res)
    models = [
        ModelSpec("r50_a", "resnet50", zoo.resnet(50, 1000), frames, chw),
        ModelSpec("r50_b", "resnet50", zoo.resnet(50, 20), frames, chw),
        ModelSpec("vgg16_a", "vgg16", zoo.vgg(16, 1000, res), frames, chw),
        ModelSpec("vgg16_b", "vgg16", zoo.vgg(16, 10, res), frames, chw),
    ]
    groups = share_by_name(models, [0, 1], _resnet_prefix([1, 2, 3]))
    groups += share_by_name(models, [2, 3],
                            lambda n: n.startswith("features."))
    return Workload("r50x2_vgg16x2", 2, "bf16", models, groups, "normal")


def yolov3x3(res=416, frames=4):
    chw = (3, res, res)
    models = [ModelSpec(f"yolov3_{c}", "yolov3", zoo.yolov3(80), frames, chw)
              for c in "abc"]
    groups = share_by_name(models, [0, 1, 2],
                           lambda n: n.startswith("backbone."))
    # the per-model heads sit 53..75 convs deep: their activations are kept
    # as bf16 pairs (about 16 significant bits), which holds the outputs'
    # drift from the float32 result well inside the bf16 tolerance
    return Workload("yolov3x3", 3, "bf16", models, groups, "uniform",
                    options={"PAIRED_ACTS": 1})


def mix8_budget40(res=224, frames=8, budget_frac=0.4):
    chw = (3, res, res)
    models = [ModelSpec(f"r152_{c}", "resnet152", zoo.resnet(152), frames, chw)
              for c in "ab"]
    models += [ModelSpec(f"r50_{c}", "resnet50", zoo.resnet(50), frames, chw)
               for c in "abc"]
    models += [ModelSpec(f"vgg19_{c}", "vgg19", zoo.vgg(19, 1000, res), frames,
                         chw) for c in "abc"]
    groups = share_by_name(models, [0, 1, 2, 3, 4], _resnet_prefix([1]))
    groups += share_by_name(models, [0, 1], lambda n: n.startswith("layer2."))
    groups += share_by_name(models, [2, 3, 4],
                            lambda n: n.startswith("layer2."))
    vgg_shared = {f"features.conv{i}" for i in range(8)} | \
        {f"features.pool{i}" for i in range(3)}
    groups += share_by_name(models, [5, 6, 7], lambda n: n in vgg_shared)
    return Workload("mix8_budget40", 4, "bf16", models, groups, "normal",
                    budget_frac)


WORKLOADS = {"tiny2": tiny2, "resnet18x2": resnet18x2,
             "r50x2_vgg16x2": r50x2_vgg16x2, "yolov3x3": yolov3x3,
             "mix8_budget40": mix8_budget40}


def get(name, **kw):
    return WORKLOADS[name](**kw)
