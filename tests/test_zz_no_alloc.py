"""The allocation-free round (gemel_infer_noalloc) through the C ABI against
gemel_infer on the same context settings: two calls in a row, the second
with fewer frames, each bitwise equal to gemel_infer's outputs (plan-time
tuning off in both, so both take the cost model's tile configurations and
sum in the same order) and within the bf16 tolerance of the oracle."""

import numpy as np
import pytest

from harness import GpuWorkload, compare, log, oracle_outputs
from workloads import configs

pytestmark = pytest.mark.gpu


def _outputs(ctx, ids, frames, noalloc):
    import torch
    dev = [torch.from_numpy(np.ascontiguousarray(f)).cuda() for f in frames]
    s = torch.cuda.Stream()
    outs = ctx.alloc_outputs(ids, [f.shape[0] for f in frames])
    with torch.cuda.stream(s):
        ctx.infer(ids, dev, stream=s, outputs=outs, noalloc=noalloc)
    s.synchronize()
    return [[o.cpu().numpy() for o in m] for m in outs]


@pytest.mark.parametrize("name,kw,small", [
    ("resnet18x2", {}, 2),
    ("yolov3x3", {"res": 160, "frames": 2}, 1),
    ("r50x2_vgg16x2", {"res": 96, "frames": 2}, 1),
])
def test_noalloc_matches_infer_on_two_calls(name, kw, small):
    from paper_2201_07705_amd import gemel as G
    wl = configs.get(name, **kw)
    wl.options = dict(wl.options, TUNE=0)
    params = [wl.params(i) for i in range(len(wl.models))]
    full = [wl.frames(i) for i in range(len(wl.models))]
    part = [f[:small] for f in full]
    ref = GpuWorkload(wl, params)
    try:
        want = [_outputs(ref.ctx, ref.ids, fr, False) for fr in (full, part)]
    finally:
        ref.close()
    g = GpuWorkload(wl, params)
    try:
        # the weights are placed by one ordinary round; the next calls
        # allocate nothing
        _outputs(g.ctx, g.ids, part, False)
        got = []
        for fr in (full, part):
            log(f"{name}: gemel_infer_noalloc on {fr[0].shape[0]} frames per model")
            got.append(_outputs(g.ctx, g.ids, fr, True))
            assert g.ctx.query(G.Q_ROUND_MODE) == 4   # caller's stream only
        # an ordinary round after them still matches
        again = _outputs(g.ctx, g.ids, full, False)
    finally:
        g.close()
    for w, o in zip(want, got):
        for a, b in zip(w, o):
            for x, y in zip(a, b):
                assert np.array_equal(x, y)
    for a, b in zip(want[0], again):
        for x, y in zip(a, b):
            assert np.array_equal(x, y)
    for fr, o in zip((full, part), got):
        compare(wl, o, oracle_outputs(wl, params, fr),
                tag=f"{name}-noalloc-{fr[0].shape[0]}")


def test_noalloc_refuses_rounds_beyond_the_static_scratch():
    """The full-size workload's activations (8 frames per model; VGG-16's
    first convs alone write 103 MB) exceed the 64 MiB static array: the
    call returns EBUDGET and enqueues nothing; an ordinary round still
    runs."""
    from paper_2201_07705_amd import gemel as G
    wl = configs.r50x2_vgg16x2()
    params = [wl.params(i) for i in range(len(wl.models))]
    fr = [wl.frames(i) for i in range(len(wl.models))]
    g = GpuWorkload(wl, params)
    try:
        _outputs(g.ctx, g.ids, fr, False)
        with pytest.raises(G.GemelError) as e:
            _outputs(g.ctx, g.ids, fr, True)
        assert e.value.code == G.EBUDGET and "static scratch" in str(e.value)
        _outputs(g.ctx, g.ids, fr, False)
    finally:
        g.close()
