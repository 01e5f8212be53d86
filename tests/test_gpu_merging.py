"""Every candidate group of a workload merged at once, on the GPU.

gemel_enumerate_groups lists all appearances of each architecturally
identical layer (Section 5.3); installing all of them makes one weight copy
serve layers at different positions of one model and at different spatial
sizes (VGG-19's 512->512 convs at 8x8 and 4x4, ResNet-34's repeated blocks),
which the plan runs as separate launches over the one copy. The outputs must
match the oracle evaluated with the same effective weights (each member
takes its group's first member's parameters)."""

import pytest

from harness import GpuWorkload, compare, log, oracle_outputs
from oracle import merging as OM
from workloads import configs, zoo

pytestmark = pytest.mark.gpu


def _variants_workload(res=64, frames=2):
    chw = (3, res, res)
    models = [configs.ModelSpec("r18", "resnet18", zoo.resnet(18), frames, chw),
              configs.ModelSpec("r34", "resnet34", zoo.resnet(34), frames, chw),
              configs.ModelSpec("v16", "vgg16", zoo.vgg(16, 1000, res), frames, chw),
              configs.ModelSpec("v19", "vgg19", zoo.vgg(19, 1000, res), frames, chw)]
    groups = [m for _, m in OM.candidate_groups(
        [(i, m.layers, m.in_chw) for i, m in enumerate(models)], 2)]
    return configs.Workload("variants", 7, "bf16", models, groups, "normal")


def test_all_candidate_groups_merged_match_oracle():
    wl = _variants_workload()
    # heterogeneous groups exist: a weight copy used at several spatial sizes
    sizes = {}
    for gi, g in enumerate(wl.groups):
        for mi, li in g:
            sh = OM.output_shapes(wl.models[mi].layers, wl.models[mi].in_chw)
            src = wl.models[mi].layers[li]["src0"]
            hw = wl.models[mi].in_chw[1:] if src < 0 else sh[src][1:]
            sizes.setdefault(gi, set()).add(tuple(hw))
    assert any(len(v) > 1 for v in sizes.values())
    params = [wl.params(i) for i in range(len(wl.models))]
    frames = [wl.frames(i) for i in range(len(wl.models))]
    log(f"variants: {len(wl.groups)} groups")
    g = GpuWorkload(wl, params)
    try:
        got = g.run(frames, repeat=2)
        # the library lists the same groups for the registered models
        lib_groups = [m for _, m in g.ctx.enumerate_groups(g.ids)]
        assert lib_groups == [[(g.ids[a], b) for a, b in gr] for gr in wl.groups]
    finally:
        g.close()
    compare(wl, got, oracle_outputs(wl, params, frames), tag="variants-64px")


def _run(wl, params, frames, **opts):
    from paper_2201_07705_amd import gemel as G
    g = GpuWorkload(wl, params)
    try:
        for k, v in opts.items():
            g.ctx.set_option(getattr(G, k), v)
        out = g.run(frames, repeat=2)
        return out, g.ctx.query(G.Q_LAUNCHES)
    finally:
        g.close()


@pytest.mark.parametrize("tile", [11, 18, 19])
def test_mixed_size_launch_equals_one_launch_per_size(tile):
    """Members of a merged group whose inputs differ in size (VGG-16's
    conv5_1 at 4x4 with VGG-19's conv4_4 at 8x8, once pooling is not fused
    into them) run as one launch whose segments keep their own sizes; with
    the tile and split-K pinned, the bits equal one launch per size."""
    import numpy as np
    wl = _variants_workload()
    params = [wl.params(i) for i in range(len(wl.models))]
    frames = [wl.frames(i) for i in range(len(wl.models))]
    log(f"mixed sizes tile {tile}")
    pin = dict(OPT_FUSE_POOL=0, OPT_CONV_TILE=tile, OPT_CONV_SPLITS=1)
    a, na = _run(wl, params, frames, OPT_MIXED_SIZES=0, **pin)
    b, nb = _run(wl, params, frames, OPT_MIXED_SIZES=1, **pin)
    assert nb < na
    for x, y in zip(a, b):
        for u, v in zip(x, y):
            assert np.array_equal(u, v)
    compare(wl, b, oracle_outputs(wl, params, frames), tag=f"variants-mixed-{tile}")


def _many_tiny(n, dtype):
    chw = (3, 24, 24)
    models = [configs.ModelSpec(f"t{i}", "tiny", zoo.tiny(10), 1 + i % 3, chw)
              for i in range(n)]
    groups = configs.share_by_name(models, list(range(n)),
                                   lambda name: name in ("conv1", "conv2"))
    return configs.Workload(f"tiny{n}", 9, dtype, models, groups, "uniform")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_more_members_than_one_launch_holds(dtype):
    """18 small CNNs share their first two convs: a merged layer has more
    members than one launch's segment table holds (16), so it runs as
    several launches over the one weight copy, and the input packs go 16
    models at a time. Ragged frame counts (1-3 per model). Every output
    against the oracle; with the tile pinned, bitwise equal to running
    every merged layer per model."""
    import numpy as np
    from paper_2201_07705_amd import gemel as G
    wl = _many_tiny(18, dtype)
    params = [wl.params(i) for i in range(len(wl.models))]
    fr = [wl.frames(i) for i in range(len(wl.models))]
    log(f"18 merged members, {dtype}")
    outs, launches = [], []
    for split in (0, 1):
        g = GpuWorkload(wl, params)
        try:
            if dtype == "bf16":
                g.ctx.set_option(G.OPT_CONV_TILE, 2)
                g.ctx.set_option(G.OPT_CONV_SPLITS, 1)
            g.ctx.set_option(G.OPT_SPLIT_MERGED, split)
            outs.append(g.run(fr))
            launches.append(g.ctx.query(G.Q_LAUNCHES))
        finally:
            g.close()
    assert launches[0] < launches[1], launches
    compare(wl, outs[0], oracle_outputs(wl, params, fr), tag=f"tiny18-{dtype}")
    for a, b in zip(outs[0], outs[1]):
        for x, y in zip(a, b):
            assert np.array_equal(x, y)
