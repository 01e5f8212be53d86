"""Rounds enqueued directly over several streams (GEMEL_OPT_STREAMS > 1,
graph replay off): independent layers are forked onto worker streams with
event waits for cross-stream dependencies. Outputs must equal the
single-stream round bitwise, with the kernel configuration pinned."""

import numpy as np
import pytest

from harness import GpuWorkload, log
from paper_2201_07705_amd import gemel as G
from workloads import configs

pytestmark = pytest.mark.gpu


def _run(wl, params, frames, repeat=1, **opts):
    g = GpuWorkload(wl, params)
    try:
        g.ctx.set_option(G.OPT_CONV_TILE, 2)
        g.ctx.set_option(G.OPT_CONV_SPLITS, 2)
        g.ctx.set_option(G.OPT_USE_GRAPH, 0)
        for k, v in opts.items():
            g.ctx.set_option(getattr(G, k), v)
        return g.run(frames, repeat=repeat)
    finally:
        g.close()


def test_eager_streams_bitwise():
    wl = configs.r50x2_vgg16x2(res=64, frames=2)
    params = [wl.params(i) for i in range(4)]
    frames = [wl.frames(i) for i in range(4)]
    log("eager streams 1 vs 4")
    base = _run(wl, params, frames, OPT_STREAMS=1)
    for ns in (4, 8):
        got = _run(wl, params, frames, repeat=2, OPT_STREAMS=ns)
        for x, y in zip(base, got):
            for u, v in zip(x, y):
                assert np.array_equal(u, v), ns
