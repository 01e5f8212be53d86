"""SLA batch sizes of a round-robin schedule (Section 3.2: per-model batch
sizes maximising the minimum per-model throughput under a per-frame
deadline, loading pipelined with inference; Section 6.1: 100 ms).

CPU: gemel_sla_batches (a host computation in libgemel) equals the
brute-force oracle (oracle/batching.py) on random and hand-worked cost
tables, batch list for batch list. GPU: gemel_profile_batches measures the
cost table of each model alone; the choice made from it equals the
oracle's on the same table, and the chosen cycle, run on the device,
takes the time the table predicts."""

import random
import time

import numpy as np
import pytest

from oracle import batching as B
from paper_2201_07705_amd import gemel as G


def _table(rng, n, nb, dup=False):
    rows = []
    for _ in range(n):
        if dup and rows:
            rows.append(list(rows[0]))
            continue
        acc, row = rng.uniform(0.5, 20), []
        for _ in range(nb):
            acc += rng.choice([0.0, rng.uniform(0.1, 9)])
            row.append(round(acc, 3))
        rows.append(row)
    return rows


def _check(cost, swap, sla, fps, pipe):
    want = B.best_batches(cost, swap, sla, fps, len(cost[0]), pipe)
    if want is None:
        with pytest.raises(G.GemelError) as e:
            G.sla_batches(cost, sla, fps, swap, pipe)
        assert e.value.code == G.EBUDGET
        return None
    got = G.sla_batches(cost, sla, fps, swap, pipe)
    assert got[0] == want[0], (cost, swap, sla, fps, pipe, got, want)
    assert got[1] == pytest.approx(want[1], rel=1e-12)
    assert got[2] == pytest.approx(want[2], rel=1e-12)
    return got


@pytest.mark.parametrize("seed", range(60))
def test_sla_batches_equal_the_oracle(seed):
    rng = random.Random(seed)
    n = rng.randint(1, 4)
    nb = {1: 12, 2: 9, 3: 6, 4: 5}[n]
    cost = _table(rng, n, nb, dup=seed % 5 == 0)
    swap = None if seed % 3 == 0 else [round(rng.uniform(0, 25), 2)
                                       for _ in range(n)]
    for sla in (40.0, 100.0, 250.0):
        for fps in (30.0, 90.0, 1e6):
            _check(cost, swap, sla, fps, seed % 2 == 0)


def test_sla_batches_hand_worked():
    cost = [[10.0, 14.0, 18.0, 22.0], [20.0, 30.0, 40.0, 50.0]]
    assert _check(cost, None, 100.0, 1000.0, True)[0] == [3, 3]
    assert _check(cost, None, 100.0, 45.0, True)[0] == [2, 2]
    assert _check(cost, [45.0, 5.0], 100.0, 1000.0, True)[0] == [2, 2]
    assert _check(cost, [45.0, 5.0], 100.0, 1000.0, False)[0] == [1, 1]


def test_sla_batches_rejects_bad_tables():
    L = G.lib()
    import ctypes
    good = [[1.0, 2.0], [1.0, 3.0]]
    for cost, sla, fps in (([[2.0, 1.0]], 100.0, 30.0),          # decreasing
                           ([[float("nan"), 1.0]], 100.0, 30.0),
                           ([[-1.0, 1.0]], 100.0, 30.0),
                           (good, 0.0, 30.0), (good, 100.0, 0.0),
                           (good, float("inf"), 30.0)):
        with pytest.raises(G.GemelError) as e:
            G.sla_batches(cost, sla, fps)
        assert e.value.code == G.EINVAL
    with pytest.raises(G.GemelError) as e:
        G.sla_batches(good, 100.0, 30.0, swap_ms=[1.0, -2.0])
    assert e.value.code == G.EINVAL
    b = (ctypes.c_int32 * 2)()
    assert L.gemel_sla_batches(0, 2, None, None, 1, 100.0, 30.0, b, None,
                               None) == G.EINVAL
    assert L.gemel_sla_batches(2, 2, None, None, 1, 100.0, 30.0, b, None,
                               None) == G.EINVAL
    # nothing meets the deadline: EBUDGET, outputs untouched
    b[0] = b[1] = 7
    flat = (ctypes.c_double * 4)(60.0, 70.0, 60.0, 70.0)
    assert L.gemel_sla_batches(2, 2, flat, None, 1, 100.0, 30.0, b, None,
                               None) == G.EBUDGET
    assert list(b) == [7, 7]


@pytest.mark.gpu
def test_profiled_schedule_on_the_device():
    """The four models of r50x2_vgg16x2 at full size, batches 1..8: the
    measured table is nondecreasing; the choice under a deadline that
    binds and an uncapped frame rate equals the oracle's on that table, is
    deadline-bound (a larger batch for any model would miss it); running
    the chosen cycle (one round per model with its batch) takes the
    predicted cycle time within 25%."""
    import torch
    from harness import GpuWorkload, log
    from workloads import configs
    wl = configs.r50x2_vgg16x2(frames=1)
    g = GpuWorkload(wl)
    try:
        t0 = time.time()
        cost = g.ctx.profile_batches(g.ids, 8, reps=5)
        log(f"profiled 4 models x 8 batches in {time.time() - t0:.1f} s")
        for row in cost:
            log("cost ms " + " ".join(f"{c:.3f}" for c in row))
            assert all(a <= b for a, b in zip(row, row[1:]))
            assert row[0] > 0
        # a deadline that binds: halfway between what batches of one and
        # batches of eight need
        fps = 1e6
        top = B.cycle_ms(cost, None, [8] * 4) + max(r[7] for r in cost)
        low = B.cycle_ms(cost, None, [1] * 4) + max(r[0] for r in cost)
        sla = 0.5 * (low + top)
        want = B.best_batches(cost, None, sla, fps, 8)
        assert want is not None
        got = G.sla_batches(cost, sla, fps)
        assert got[0] == want[0]
        log(f"batches {got[0]}, {got[1]:.0f} frames/s per model, "
            f"cycle {got[2]:.3f} ms")
        b = got[0]
        # deadline-bound: growing any model's batch misses the deadline or
        # exceeds the table
        for m in range(4):
            if b[m] < 8:
                up = list(b)
                up[m] += 1
                assert not B.feasible(cost, None, up, sla) or \
                    B.min_throughput(cost, None, up, fps) <= got[1]
        # the chosen cycle on the device
        frames = [torch.zeros((8,) + tuple(m.in_chw), dtype=torch.float32,
                              device="cuda") for m in wl.models]
        s = torch.cuda.Stream()
        outs = {}
        with torch.cuda.stream(s):
            def cycle():
                for m in range(4):
                    fr = frames[m][:b[m]]
                    outs[m] = g.ctx.infer([g.ids[m]], [fr], stream=s,
                                          outputs=outs.get(m))
            for _ in range(30):        # plans, tuning
                cycle()
            s.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), \
                torch.cuda.Event(enable_timing=True)
            e0.record(s)
            for _ in range(20):
                cycle()
            e1.record(s)
        s.synchronize()
        ms = e0.elapsed_time(e1) / 20
        log(f"measured cycle {ms:.3f} ms, predicted {got[2]:.3f} ms")
        assert ms <= 1.25 * got[2] and ms >= 0.75 * got[2]
        assert np.isfinite(outs[0][0][0].cpu().numpy()).all()
    finally:
        g.close()
