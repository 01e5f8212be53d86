"""Architecture descriptors of the vision CNNs in the merged workloads.

Pure data: each builder returns a list of layer dicts in topological order
(every ``src0``/``src1``/``res`` index is smaller than the layer's own
index). Nothing here computes anything of the method; the dicts are what a
user hands to ``gemel_register_model`` and what the oracle walks.

Layer dict keys
---------------
name      unique dotted name inside the model (``layer1.0.conv1``)
op        'conv' | 'fc' | 'maxpool' | 'avgpool' | 'upsample' | 'concat'
src0      producer layer index, -1 = model input
src1      second producer (concat only), else -1
cin,cout  channels (fc: flattened input features / output features)
kh,kw,stride,pad   window (conv, maxpool)
act       'none' | 'relu' | 'leaky'   (leaky slope 0.1)
res       index of a layer whose output is added, -1 = none
res_mode  'add_act' (y = act(z + r), ResNet) | 'act_add' (y = act(z) + r,
          Darknet)
bias      conv/fc has a bias vector
bn        conv is followed by a batch-norm layer (running statistics)
out       the layer's output is a model output

The architectures follow the published definitions of ResNet v1.5 (stride on
the bottleneck 3x3 conv), torchvision-style VGG, Darknet-53 and the YOLOv3
three-scale head; the paper uses these model families (Table 1, Section 2
workloads) without restating their definitions.
"""

from __future__ import annotations

OPS = ("conv", "fc", "maxpool", "avgpool", "upsample", "concat")


def _layer(name, op, src0, **kw):
    d = dict(name=name, op=op, src0=src0, src1=-1, cin=0, cout=0, kh=1, kw=1,
             stride=1, pad=0, act="none", res=-1, res_mode="add_act",
             bias=False, bn=False, out=False)
    d.update(kw)
    return d


class _Builder:
    def __init__(self):
        self.layers = []

    def add(self, name, op, src0, **kw):
        self.layers.append(_layer(name, op, src0, **kw))
        return len(self.layers) - 1

    def conv(self, name, src, cin, cout, k, stride=1, pad=None, act="relu",
             bn=True, bias=False, res=-1, res_mode="add_act", out=False):
        if pad is None:
            pad = k // 2
        return self.add(name, "conv", src, cin=cin, cout=cout, kh=k, kw=k,
                        stride=stride, pad=pad, act=act, bn=bn, bias=bias,
                        res=res, res_mode=res_mode, out=out)


def tiny(classes=10):
    """Two shared-able 3x3 convs, a 3x3 head conv, global avgpool, FC."""
    b = _Builder()
    x = b.conv("conv1", -1, 3, 16, 3, 1, 1, bn=False, bias=True)
    x = b.conv("conv2", x, 16, 32, 3, 2, 1, bn=False, bias=True)
    x = b.conv("head.conv", x, 32, 32, 3, 1, 1, bn=False, bias=True)
    x = b.add("head.pool", "avgpool", x, cin=32, cout=32)
    b.add("head.fc", "fc", x, cin=32, cout=classes, bias=True, out=True)
    return b.layers


_RESNET_BLOCKS = {18: ("basic", [2, 2, 2, 2]), 34: ("basic", [3, 4, 6, 3]),
                  50: ("bottleneck", [3, 4, 6, 3]),
                  101: ("bottleneck", [3, 4, 23, 3]),
                  152: ("bottleneck", [3, 8, 36, 3])}


def resnet(depth, classes=1000):
    kind, counts = _RESNET_BLOCKS[depth]
    exp = 1 if kind == "basic" else 4
    b = _Builder()
    x = b.conv("conv1", -1, 3, 64, 7, 2, 3)
    x = b.add("maxpool", "maxpool", x, cin=64, cout=64, kh=3, kw=3, stride=2,
              pad=1)
    cin = 64
    for si, (width, n) in enumerate(zip([64, 128, 256, 512], counts)):
        for bi in range(n):
            stride = 2 if (bi == 0 and si > 0) else 1
            p = f"layer{si + 1}.{bi}"
            cout = width * exp
            if kind == "basic":
                y = b.conv(p + ".conv1", x, cin, width, 3, stride)
                short = x
                if stride != 1 or cin != cout:
                    short = b.conv(p + ".downsample", x, cin, cout, 1, stride,
                                   act="none")
                x = b.conv(p + ".conv2", y, width, cout, 3, 1, res=short)
            else:
                y = b.conv(p + ".conv1", x, cin, width, 1, 1)
                y = b.conv(p + ".conv2", y, width, width, 3, stride)
                short = x
                if stride != 1 or cin != cout:
                    short = b.conv(p + ".downsample", x, cin, cout, 1, stride,
                                   act="none")
                x = b.conv(p + ".conv3", y, width, cout, 1, 1, res=short)
            cin = cout
    x = b.add("avgpool", "avgpool", x, cin=cin, cout=cin)
    b.add("fc", "fc", x, cin=cin, cout=classes, bias=True, out=True)
    return b.layers


_VGG_CFG = {
    11: [64, "M", 128, "M", 256, 256, "M", 512, 512, "M", 512, 512, "M"],
    16: [64, 64, "M", 128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M",
         512, 512, 512, "M"],
    19: [64, 64, "M", 128, 128, "M", 256, 256, 256, 256, "M", 512, 512, 512,
         512, "M", 512, 512, 512, 512, "M"],
}


def vgg(depth, classes=1000, in_hw=224):
    """torchvision-style VGG without BN. At 224x224 input the adaptive 7x7
    average pool is the identity and is omitted; dropout is inference-off.
    Other input sizes (multiples of 32) flatten (in_hw/32)^2 positions into
    FC6 instead of 7x7."""
    b = _Builder()
    x, cin, ci, pi = -1, 3, 0, 0
    for v in _VGG_CFG[depth]:
        if v == "M":
            x = b.add(f"features.pool{pi}", "maxpool", x, cin=cin, cout=cin,
                      kh=2, kw=2, stride=2, pad=0)
            pi += 1
        else:
            x = b.conv(f"features.conv{ci}", x, cin, v, 3, 1, 1, bn=False,
                       bias=True)
            cin, ci = v, ci + 1
    s = in_hw // 32
    x = b.add("classifier.fc6", "fc", x, cin=512 * s * s, cout=4096,
              bias=True, act="relu")
    x = b.add("classifier.fc7", "fc", x, cin=4096, cout=4096, bias=True,
              act="relu")
    b.add("classifier.fc8", "fc", x, cin=4096, cout=classes, bias=True,
          out=True)
    return b.layers


def _darknet53(b):
    """Darknet-53 feature extractor (52 convs). Returns (out, tap26, tap52):
    the 13x13x1024 output and the 26x26x512 / 52x52x256 route taps."""
    lk = dict(act="leaky")
    x = b.conv("backbone.conv0", -1, 3, 32, 3, **lk)
    cin = 32
    taps = {}
    for si, (cout, n) in enumerate(zip([64, 128, 256, 512, 1024],
                                       [1, 2, 8, 8, 4])):
        x = b.conv(f"backbone.down{si}", x, cin, cout, 3, 2, 1, **lk)
        for bi in range(n):
            p = f"backbone.stage{si}.{bi}"
            y = b.conv(p + ".conv1", x, cout, cout // 2, 1, **lk)
            x = b.conv(p + ".conv2", y, cout // 2, cout, 3, res=x,
                       res_mode="act_add", **lk)
        cin = cout
        taps[cout] = x
    return x, taps[512], taps[256]


def yolov3(classes=80):
    """Darknet-53 backbone + the three-scale YOLOv3 head (75 convs)."""
    b = _Builder()
    lk = dict(act="leaky")
    outc = 3 * (classes + 5)
    x, tap26, tap52 = _darknet53(b)
    cin = 1024
    for hi, (w, tap) in enumerate([(512, None), (256, tap26), (128, tap52)]):
        p = f"head{hi}"
        if tap is not None:
            r = b.conv(p + ".route", route_src, route_c, w, 1, **lk)
            u = b.add(p + ".upsample", "upsample", r, cin=w, cout=w)
            tap_c = b.layers[tap]["cout"]
            x = b.add(p + ".concat", "concat", u, src1=tap, cin=w,
                      cout=w + tap_c)
            cin = w + tap_c
        for j in range(5):
            k, c = (1, w) if j % 2 == 0 else (3, 2 * w)
            x = b.conv(f"{p}.conv{j}", x, cin, c, k, **lk)
            cin = c
        route_src, route_c = x, w
        y = b.conv(p + ".conv5", x, w, 2 * w, 3, **lk)
        b.conv(p + ".out", y, 2 * w, outc, 1, act="none", bn=False, bias=True,
               out=True)
    return b.layers


def build(arch):
    """Builder lookup by architecture name ('resnet50', 'vgg16', ...)."""
    if arch == "tiny":
        return tiny()
    if arch.startswith("resnet"):
        return resnet(int(arch[6:]))
    if arch.startswith("vgg"):
        return vgg(int(arch[3:]))
    if arch == "yolov3":
        return yolov3()
    raise KeyError(arch)


def with_classes(layers, classes):
    """Copy of a classifier's layer list with its last FC resized."""
    out = [dict(l) for l in layers]
    last = out[-1]
    assert last["op"] in ("fc", "conv") and last["out"]
    last["cout"] = classes
    return out


# ---- shape and size bookkeeping (data about the inputs, no arithmetic of
# the method itself) ----

def shapes(layers, in_chw):
    """Per-layer output (C, H, W) for a model input of shape in_chw."""
    out = []
    for l in layers:
        src = in_chw if l["src0"] < 0 else out[l["src0"]]
        c, h, w = src
        op = l["op"]
        if op == "conv" or op == "maxpool":
            ho = (h + 2 * l["pad"] - l["kh"]) // l["stride"] + 1
            wo = (w + 2 * l["pad"] - l["kw"]) // l["stride"] + 1
            out.append((l["cout"], ho, wo))
        elif op == "avgpool":
            out.append((c, 1, 1))
        elif op == "fc":
            out.append((l["cout"], 1, 1))
        elif op == "upsample":
            out.append((c, 2 * h, 2 * w))
        elif op == "concat":
            c1 = out[l["src1"]][0]
            out.append((c + c1, h, w))
        else:
            raise ValueError(op)
    return out


def param_count(layers):
    """Trainable parameters as frameworks count them: conv/fc weights and
    biases, plus BN gamma and beta (running statistics are buffers)."""
    n = 0
    for l in layers:
        if l["op"] == "conv":
            n += l["cout"] * l["cin"] * l["kh"] * l["kw"]
        elif l["op"] == "fc":
            n += l["cout"] * l["cin"]
        else:
            continue
        if l["bias"]:
            n += l["cout"]
        if l["bn"]:
            n += 2 * l["cout"]
    return n


def layer_param_count(l):
    return param_count([l])


def macs(layers, in_chw):
    """Multiply-accumulates of one frame through conv and FC layers."""
    sh = shapes(layers, in_chw)
    n = 0
    for l, (c, h, w) in zip(layers, sh):
        if l["op"] == "conv":
            n += c * h * w * l["cin"] * l["kh"] * l["kw"]
        elif l["op"] == "fc":
            n += l["cout"] * l["cin"]
    return n
