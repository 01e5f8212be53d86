"""Layer-level parity of the HIP kernels against the oracle, through the C
ABI: single conv/FC/pool/routing layers and small graphs, chosen to span
several tiles, ragged M/N/K tails, split-K, padded channel counts, both
residual orders, the NHWC internal store and the NCHW fp32 output store,
and merged launches whose segments carry different frame counts."""

import numpy as np
import pytest

from harness import GpuWorkload, compare, log, oracle_outputs
from workloads.configs import ModelSpec, Workload

pytestmark = pytest.mark.gpu

BF16_LAYER_TOL = 1e-2   # one or two bf16 roundings of the activations
F32_LAYER_TOL = 1e-4


def L(name, op, src0, **kw):
    d = dict(name=name, op=op, src0=src0, src1=-1, cin=0, cout=0, kh=1, kw=1,
             stride=1, pad=0, act="none", res=-1, res_mode="add_act",
             bias=False, bn=False, out=False)
    d.update(kw)
    return d


def conv(name, src, cin, cout, k, s=1, p=0, **kw):
    return L(name, "conv", src, cin=cin, cout=cout, kh=k, kw=k, stride=s,
             pad=p, **kw)


def run_case(layers_per_model, in_chw, frames, dtype, groups=(), seed=7,
             tol=None, dist="normal", tile=-1):
    models = [ModelSpec(f"m{i}", "custom", lay, n, in_chw)
              for i, (lay, n) in enumerate(zip(layers_per_model, frames))]
    wl = Workload(f"case{seed}", seed, dtype, models, list(groups), dist)
    params = [wl.params(i) for i in range(len(models))]
    fr = [wl.frames(i) for i in range(len(models))]
    g = GpuWorkload(wl, params)
    try:
        if tile >= 0:
            from paper_2201_07705_amd import gemel as G
            g.ctx.set_option(G.OPT_CONV_TILE, tile)
        got = g.run(fr)
    finally:
        g.close()
    ref = oracle_outputs(wl, params, fr)
    tol = tol or (BF16_LAYER_TOL if dtype == "bf16" else F32_LAYER_TOL)
    return compare(wl, got, ref, tol=tol, check_argmax=False)


CONV_CASES = [
    # cin, cout, k, stride, pad, hw, frames
    (3, 64, 7, 2, 3, 64, 2),
    (64, 64, 3, 1, 1, 20, 3),
    (64, 256, 1, 1, 0, 14, 2),
    (128, 96, 3, 2, 1, 15, 2),
    (256, 255, 1, 1, 0, 13, 2),
    (512, 512, 3, 1, 1, 7, 2),
    (32, 64, 3, 2, 1, 33, 1),
    (16, 40, 3, 1, 1, 9, 5),
    (1024, 64, 1, 1, 0, 5, 3),
    # 8-channel (RGB stem) inputs: narrow N, ragged M, N beyond one tile
    (3, 32, 3, 1, 1, 41, 3),
    (3, 64, 3, 1, 1, 30, 2),
    (8, 40, 5, 2, 2, 23, 2),
    (3, 96, 3, 2, 1, 17, 1),
]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("case", CONV_CASES, ids=lambda c: "x".join(map(str, c)))
def test_conv_layer_output_store(dtype, case):
    cin, cout, k, s, p, hw, n = case
    log(f"conv {case} {dtype}")
    lay = [conv("c", -1, cin, cout, k, s, p, bias=True, act="relu", out=True)]
    run_case([lay], (cin, hw, hw), [n], dtype)


TILES = ["128x128", "128x64", "64x64", "256x256", "256x128", "256x64",
         "64x64d2", "128x64d2", "64x128", "dma256x256", "dma256x128",
         "dma128x128", "dma128x64", "stem", "dma64_256x256", "dma64_256x128",
         "dma64_128x128", "dma64_128x64", "dma64x64", "dma64_64x64",
         "dma256x128w8", "dma128x256w8", "dma256x64", "dma64x256"]


@pytest.mark.parametrize("tile", range(len(TILES)), ids=lambda t: TILES[t])
@pytest.mark.parametrize("case", CONV_CASES, ids=lambda c: "x".join(map(str, c)))
def test_conv_every_tile_shape(tile, case):
    """Every tile shape (forced) on every conv case, internal bf16 store
    with a residual and the fp32 output store."""
    cin, cout, k, s, p, hw, n = case
    log(f"tile {TILES[tile]} conv {case}")
    lay = [conv("c", -1, cin, cout, k, s, p, bn=True, act="leaky"),
           conv("d", 0, cout, cout, 1, 1, 0, bn=True, act="relu", res=0),
           conv("o", 1, cout, 24, 3, 1, 1, bias=True, out=True)]
    run_case([lay], (cin, hw, hw), [n], "bf16", tile=tile)


# One conv written straight to the fp32 output: inputs and weights are
# bf16-exact and accumulation is fp32, so the only difference from the fp64
# oracle is fp32 summation order (relative error ~ sqrt(K) * 2^-24 of the
# terms' magnitude).
EXACT_TOL = 5e-5


@pytest.mark.parametrize("splits,fused", [(1, 0), (3, 0), (3, 2)],
                         ids=["split1", "split3", "split3fused"])
@pytest.mark.parametrize("tile", range(len(TILES)), ids=lambda t: TILES[t])
@pytest.mark.parametrize("case", CONV_CASES, ids=lambda c: "x".join(map(str, c)))
def test_conv_single_layer_exact(tile, case, splits, fused):
    """Every tile shape and split-K 1/3 (partial sums reduced by a separate
    launch or inside the GEMM launch) on one conv + BN + residual-free
    epilogue with the fp32 output store, against the oracle at fp32
    accumulation precision."""
    from paper_2201_07705_amd import gemel as G
    cin, cout, k, s, p, hw, n = case
    log(f"exact tile {TILES[tile]} splits {splits} conv {case}")
    lay = [conv("c", -1, cin, cout, k, s, p, bn=True, act="leaky", out=True)]
    models = [ModelSpec("m0", "custom", lay, n, (cin, hw, hw))]
    wl = Workload("exact", 11, "bf16", models, [], "normal")
    params = [wl.params(0)]
    fr = [wl.frames(0)]
    g = GpuWorkload(wl, params)
    try:
        g.ctx.set_option(G.OPT_CONV_TILE, tile)
        g.ctx.set_option(G.OPT_CONV_SPLITS, splits)
        g.ctx.set_option(G.OPT_SPLITK_FUSED, fused)
        got = g.run(fr)
    finally:
        g.close()
    compare(wl, got, oracle_outputs(wl, params, fr), tol=EXACT_TOL,
            check_argmax=False)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("case", CONV_CASES[:6], ids=lambda c: "x".join(map(str, c)))
def test_conv_layer_internal_store_and_export(dtype, case):
    cin, cout, k, s, p, hw, n = case
    log(f"conv+export {case} {dtype}")
    lay = [conv("c", -1, cin, cout, k, s, p, bn=True, act="leaky"),
           L("copy", "maxpool", 0, cin=cout, cout=cout, kh=1, kw=1, out=True)]
    run_case([lay], (cin, hw, hw), [n], dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("act,mode", [("relu", "add_act"), ("leaky", "act_add"),
                                      ("none", "add_act")])
def test_conv_residual_orders(dtype, act, mode):
    log(f"residual {act} {mode} {dtype}")
    lay = [conv("a", -1, 32, 64, 3, 1, 1, bn=True, act="relu"),
           conv("b", 0, 64, 64, 3, 1, 1, bn=True, act=act, res=0,
                res_mode=mode),
           conv("c", 1, 64, 128, 1, 1, 0, bias=True, act="relu", out=True)]
    run_case([lay], (32, 17, 17), [3], dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("frames", [1, 3, 8, 20, 80])
def test_fc_stack_small_and_large_batches(dtype, frames):
    log(f"fc stack frames={frames} {dtype}")
    # NCHW flatten of a 64 x 7 x 7 map, two FC layers (internal + output)
    lay = [conv("c", -1, 8, 64, 3, 1, 1, bias=True, act="relu"),
           L("fc1", "fc", 0, cin=64 * 49, cout=520, bias=True, act="relu"),
           L("fc2", "fc", 1, cin=520, cout=1000, bias=True, out=True)]
    run_case([lay], (8, 7, 7), [frames], dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_pools(dtype):
    log(f"pools {dtype}")
    lay = [conv("c", -1, 3, 64, 3, 2, 1, bn=True, act="relu"),
           L("mp3", "maxpool", 0, cin=64, cout=64, kh=3, kw=3, stride=2,
             pad=1),
           L("mp2", "maxpool", 1, cin=64, cout=64, kh=2, kw=2, stride=2),
           L("gap", "avgpool", 2, cin=64, cout=64),
           L("fc", "fc", 3, cin=64, cout=10, bias=True, out=True)]
    run_case([lay], (3, 57, 57), [4], dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_upsample_concat_route(dtype):
    log(f"route {dtype}")
    lay = [conv("a", -1, 8, 32, 3, 2, 1, bn=True, act="leaky"),   # 16x16
           conv("b", 0, 32, 64, 3, 2, 1, bn=True, act="leaky"),   # 8x8
           conv("r", 1, 64, 16, 1, 1, 0, bn=True, act="leaky"),
           L("up", "upsample", 2, cin=16, cout=16),                # 16x16
           L("cat", "concat", 3, src1=0, cin=16, cout=48),
           conv("o", 4, 48, 255, 1, 1, 0, bias=True, out=True),
           conv("o2", 1, 64, 24, 3, 1, 1, bias=True, out=True)]
    run_case([lay], (8, 32, 32), [3], dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_merged_segments_with_different_frame_counts(dtype):
    log(f"merged segments {dtype}")
    body = [conv("c1", -1, 3, 32, 3, 1, 1, bn=True, act="relu"),
            conv("c2", 0, 32, 64, 3, 2, 1, bn=True, act="relu"),
            conv("c3", 1, 64, 64, 3, 1, 1, bn=True, act="relu", res=1),
            L("gap", "avgpool", 2, cin=64, cout=64)]
    heads = [L("fc", "fc", 3, cin=64, cout=c, bias=True, out=True)
             for c in (10, 37, 5)]
    models = [body + [h] for h in heads]
    groups = [[(0, i), (1, i), (2, i)] for i in range(4)]
    run_case(models, (3, 24, 24), [2, 5, 1], dtype, groups)


def _deep_chain(depth=16, c=64, with_route=True):
    """A per-model chain of 3x3 / 1x1 convs with batch norm and leaky ReLU
    (the shape of a detection head), optionally with an upsample + concat
    route, ending in a linear 1x1 output conv."""
    lay = [conv("c0", -1, 3, c, 3, 1, 1, bn=True, act="leaky")]
    for i in range(1, depth):
        k = 3 if i % 2 else 1
        lay.append(conv(f"c{i}", i - 1, c, c, k, 1, k // 2, bn=True,
                        act="leaky"))
    src = len(lay) - 1
    if with_route:
        # route: 1x1 conv, 2x2 max pool (a coarser scale), upsample, then
        # concat with the chain's own output (a paired tap next to a plain
        # bf16 tensor in one concat)
        lay.append(conv("r", src, c, c // 2, 1, bn=True, act="leaky"))
        lay.append(L("p", "maxpool", len(lay) - 1, cin=c // 2, cout=c // 2,
                     kh=2, kw=2, stride=2))
        lay.append(L("u", "upsample", len(lay) - 1, cin=c // 2, cout=c // 2))
        lay.append(L("cat", "concat", len(lay) - 1, src1=src, cin=c // 2,
                     cout=c // 2 + c))
        lay.append(conv("m", len(lay) - 1, c // 2 + c, c, 3, 1, 1, bn=True,
                        act="leaky"))
        src = len(lay) - 1
    lay.append(conv("out", src, c, 40, 1, bias=True, out=True))
    return lay


@pytest.mark.parametrize("with_route", [False, True])
def test_paired_activations_cut_drift_of_deep_unmerged_chains(with_route):
    """GEMEL_OPT_PAIRED_ACTS keeps unmerged activations as bf16 (hi, lo)
    pairs: the output of a deep per-model chain then drifts from the
    float32 oracle by far less than with bf16 activations. What remains is
    mostly the one bf16 rounding of the first conv's output (it reads the
    8-channel input and stays bf16; with the route, also the pooled route
    tensor), which the chain's gain carries to the output: about a third of
    the drift of 16 roundings or less."""
    from paper_2201_07705_amd import gemel as G
    lay = _deep_chain(with_route=with_route)
    models = [ModelSpec("m0", "custom", lay, 3, (3, 24, 24))]
    errs = {}
    for paired in (0, 1):
        wl = Workload("chain", 11, "bf16", models, [], "uniform",
                      options={"PAIRED_ACTS": paired})
        params = [wl.params(0)]
        fr = [wl.frames(0)]
        g = GpuWorkload(wl, params)
        try:
            got = g.run(fr)
        finally:
            g.close()
        errs[paired] = compare(wl, got, oracle_outputs(wl, params, fr),
                               tol=BF16_LAYER_TOL * 3, check_argmax=False,
                               tag=f"chain-pairs{paired}")
    log(f"deep chain normwise error: bf16 {errs[0]:.3e}, pairs {errs[1]:.3e}")
    assert errs[1] <= 5e-3 and errs[1] * 3 <= errs[0], errs


def test_paired_activations_leave_merged_layers_bitwise():
    """Pairs apply only to tensors between unmerged layers: on a workload
    whose every conv is merged (ResNet-18 x2, reduced), the outputs with
    and without the option are bitwise equal."""
    import numpy as np
    from workloads import configs
    wl = configs.resnet18x2(res=64, frames=2)
    params = [wl.params(i) for i in range(len(wl.models))]
    fr = [wl.frames(i) for i in range(len(wl.models))]
    outs = []
    for paired in (0, 1):
        wl.options = {"PAIRED_ACTS": paired, "TUNE": 0}
        g = GpuWorkload(wl, params)
        try:
            outs.append(g.run(fr))
        finally:
            g.close()
    for a, b in zip(outs[0], outs[1]):
        for x, y in zip(a, b):
            assert np.array_equal(x, y)


DMA_TILES = [t for t, n in enumerate(TILES) if n.startswith("dma")]
GROUP_CASES = [
    # cin, cout, k, stride, pad, hw, frames per model (ragged segments)
    (64, 64, 3, 1, 1, 13, (1, 3, 2)),
    (128, 96, 1, 1, 0, 9, (2, 1, 4)),
    (256, 255, 1, 1, 0, 13, (3, 3, 3)),
    (64, 128, 3, 2, 1, 15, (2, 5)),
]


@pytest.mark.parametrize("splits,fused", [(1, 0), (3, 0), (3, 2)],
                         ids=["split1", "split3", "split3fused"])
@pytest.mark.parametrize("tile", DMA_TILES, ids=lambda t: TILES[t])
@pytest.mark.parametrize("case", GROUP_CASES, ids=lambda c: "x".join(map(str, c[:6])))
def test_grouped_unmerged_conv_exact(tile, case, splits, fused):
    """The same unmerged conv in several models (each its own weights, BN
    and frame count; segments of ragged row counts) as ONE grouped launch:
    every LDS-DMA tile, split-K 1/3, against the oracle at fp32
    accumulation precision, and bitwise equal to one launch per model in
    the same configuration."""
    import numpy as np
    from paper_2201_07705_amd import gemel as G
    cin, cout, k, s, p, hw, frames = case
    log(f"grouped tile {TILES[tile]} splits {splits} conv {case}")
    models = [ModelSpec(f"m{i}", "custom",
                        [conv("c", -1, cin, cout, k, s, p, bn=True,
                              act="leaky", out=True)], n, (cin, hw, hw))
              for i, n in enumerate(frames)]
    wl = Workload("grouped", 13, "bf16", models, [], "normal")
    params = [wl.params(i) for i in range(len(models))]
    fr = [wl.frames(i) for i in range(len(models))]
    outs, launches = [], []
    for grouped in (1, 0):
        g = GpuWorkload(wl, params)
        try:
            g.ctx.set_option(G.OPT_GROUP_UNMERGED, grouped)
            g.ctx.set_option(G.OPT_CONV_TILE, tile)
            g.ctx.set_option(G.OPT_CONV_SPLITS, splits)
            g.ctx.set_option(G.OPT_SPLITK_FUSED, fused)
            outs.append(g.run(fr))
            launches.append(g.ctx.query(G.Q_LAUNCHES))
        finally:
            g.close()
    assert launches[0] < launches[1], launches
    compare(wl, outs[0], oracle_outputs(wl, params, fr), tol=EXACT_TOL,
            check_argmax=False)
    for a, b in zip(outs[0], outs[1]):
        for x, y in zip(a, b):
            assert np.array_equal(x, y)


@pytest.mark.parametrize("name,kw", [("r50x2_vgg16x2", {"res": 64, "frames": 2}),
                                     ("yolov3x3", {"res": 96, "frames": 2})])
def test_grouped_unmerged_workloads(name, kw):
    """Whole workloads with the per-model layers grouped (ResNet-50 layer4,
    the YOLOv3 heads): fewer launches, the oracle's outputs within the
    workload tolerance, and bitwise equal to one launch per model with the
    tile configuration forced alike."""
    import numpy as np
    from paper_2201_07705_amd import gemel as G
    from workloads import configs
    wl = configs.get(name, **kw)
    params = [wl.params(i) for i in range(len(wl.models))]
    fr = [wl.frames(i) for i in range(len(wl.models))]
    outs, launches = [], []
    for grouped in (1, 0):
        g = GpuWorkload(wl, params)
        try:
            g.ctx.set_option(G.OPT_GROUP_UNMERGED, grouped)
            g.ctx.set_option(G.OPT_CONV_TILE, 11)   # LDS-DMA 128x128
            g.ctx.set_option(G.OPT_CONV_SPLITS, 1)
            outs.append(g.run(fr))
            launches.append(g.ctx.query(G.Q_LAUNCHES))
        finally:
            g.close()
    log(f"{name}: launches grouped {launches[0]}, per model {launches[1]}")
    assert launches[0] < launches[1]
    compare(wl, outs[0], oracle_outputs(wl, params, fr), tag=f"{name}-grouped")
    for a, b in zip(outs[0], outs[1]):
        for x, y in zip(a, b):
            assert np.array_equal(x, y)


FC_GROUP_CASES = [
    # producer C x H x W, FC widths, frames per model
    ((64, 7, 7), (520, 1000), (3, 5)),
    ((512, 7, 7), (4096, 1000), (8, 8)),
    ((32, 4, 4), (264,), (20, 30, 40)),   # more than 64 frames: two nodes
]


@pytest.mark.parametrize("fused", [0, 1], ids=["reduce", "fused"])
@pytest.mark.parametrize("case", FC_GROUP_CASES, ids=lambda c: f"{c[0][0]}x{c[0][1]}-{'-'.join(map(str, c[2]))}")
def test_grouped_unmerged_fc_exact(case, fused):
    """The same unmerged FC stack in several models (each its own weights,
    bias and frame count) as grouped FC launches (one grid slice per model):
    against the oracle, and bitwise equal to one launch per model (the
    grouped launch takes one member's split configuration)."""
    import numpy as np
    from paper_2201_07705_amd import gemel as G
    (c, h, w), widths, frames = case
    log(f"grouped fc {case} fused {fused}")
    lay = [conv("c", -1, 8, c, 1, 1, 0, bias=True, act="relu")]
    k = c * h * w
    for i, n in enumerate(widths):
        lay.append(L(f"fc{i}", "fc", i, cin=k, cout=n, bias=True,
                     act="relu" if i + 1 < len(widths) else "none",
                     out=i + 1 == len(widths)))
        k = n
    models = [ModelSpec(f"m{i}", "custom", lay, n, (8, h, w))
              for i, n in enumerate(frames)]
    wl = Workload("fcgroup", 17, "bf16", models, [], "normal")
    params = [wl.params(i) for i in range(len(models))]
    fr = [wl.frames(i) for i in range(len(models))]
    outs, launches = [], []
    for grouped in (1, 0):
        g = GpuWorkload(wl, params)
        try:
            g.ctx.set_option(G.OPT_GROUP_UNMERGED, grouped)
            g.ctx.set_option(G.OPT_SPLITK_FUSED, fused)
            g.ctx.set_option(G.OPT_TUNE, 0)
            outs.append(g.run(fr))
            launches.append(g.ctx.query(G.Q_LAUNCHES))
        finally:
            g.close()
    log(f"launches grouped {launches[0]}, per model {launches[1]}")
    assert launches[0] < launches[1], launches
    compare(wl, outs[0], oracle_outputs(wl, params, fr), tol=BF16_LAYER_TOL,
            check_argmax=False, tag="fc-grouped")
    for a, b in zip(outs[0], outs[1]):
        for x, y in zip(a, b):
            assert np.array_equal(x, y)
