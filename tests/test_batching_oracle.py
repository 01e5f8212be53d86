"""Pins of the SLA batch-size oracle (oracle/batching.py; Section 3.2's
round-robin schedule whose per-model batch sizes maximise the minimum
per-model throughput under a per-frame deadline, Section 6.1's 100 ms SLA,
Section 5.4's pipelined loading) against closed forms, hand-worked cases
that separate each rule, and monotonicity on random tables."""

import math
import random

import pytest

from oracle import batching as B


def _linear(a, k, n):
    return [a + k * b for b in range(1, n + 1)]


@pytest.mark.parametrize("a,k,sla", [(5.0, 2.0, 100.0), (12.0, 0.5, 100.0),
                                     (1.0, 3.0, 40.0)])
def test_single_model_takes_the_largest_batch_within_half_the_sla(a, k, sla):
    # T = c(b), latency 2 c(b) <= SLA, b / (a + k b) grows with b
    cost = [_linear(a, k, 64)]
    b, v, t = B.best_batches(cost, None, sla, 1e9, 64)
    want = min(64, math.floor((sla / 2 - a) / k))
    assert b == [want]
    assert t == pytest.approx(a + k * want)
    assert v == pytest.approx(want / (t / 1000))


@pytest.mark.parametrize("n", [2, 3])
def test_identical_models_share_one_batch_size(n):
    # T = n c(b); latency (n + 1) c(b) <= SLA
    a, k, sla = 4.0, 1.5, 100.0
    cost = [_linear(a, k, 32) for _ in range(n)]
    b, v, t = B.best_batches(cost, None, sla, 1e9, 32)
    want = math.floor((sla / (n + 1) - a) / k)
    assert b == [want] * n
    assert t == pytest.approx(n * (a + k * want))


def test_frame_rate_caps_throughput_and_the_shorter_cycle_wins():
    # one model, c(b) = 10 + 2b ms: b / c(b) >= 30 fps first at b = 1
    # (1 / 12 ms = 83 fps), so every feasible b ties at 30 fps and the
    # shortest cycle (b = 1) is chosen
    cost = [_linear(10.0, 2.0, 20)]
    b, v, t = B.best_batches(cost, None, 100.0, 30.0, 20)
    assert b == [1] and v == 30.0 and t == 12.0
    # at 200 fps: b / (10 + 2b) ms >= 0.2 frames/ms first at b = 4 (b = 3:
    # 3 / 16 ms = 187.5 fps; b = 4: 4 / 18 ms = 222 fps)
    b, v, t = B.best_batches(cost, None, 100.0, 200.0, 20)
    assert b == [4] and v == 200.0 and t == 18.0


COST2 = [[10.0, 14.0, 18.0, 22.0], [20.0, 30.0, 40.0, 50.0]]


def test_hand_worked_two_models():
    # no swap: (3, 3) gives T = 58 ms, latency 58 + 40 = 98 <= 100 and
    # 3 / 0.058 = 51.7 fps; (4, 4) would give 55.6 fps with T = 72 <= 100
    # but its latency 72 + 50 = 122 misses the SLA
    b, v, t = B.best_batches(COST2, None, 100.0, 1000.0, 4)
    assert b == [3, 3] and t == 58.0
    assert v == pytest.approx(3 / 0.058)
    # capped at 45 fps: (2, 2) (45.5 fps) and (3, 3) tie at 45; the
    # shorter cycle (44 ms) wins
    b, v, t = B.best_batches(COST2, None, 100.0, 45.0, 4)
    assert b == [2, 2] and t == 44.0 and v == 45.0


def test_pipelined_loading_overlaps_the_next_models_swap():
    # swap = [45, 5]: pipelined, a visit to model 0 overlaps model 1's
    # load and vice versa: T = max(c0, 5) + max(c1, 45). (3, 3): T = 63,
    # latency 103 > 100. (2, 2) and (2, 3) both give T = 59 and 2 frames:
    # the lexicographically smaller (2, 2) wins
    swap = [45.0, 5.0]
    b, v, t = B.best_batches(COST2, swap, 100.0, 1000.0, 4)
    assert b == [2, 2] and t == 59.0
    assert v == pytest.approx(2 / 0.059)
    # not pipelined: T = 50 + c0 + c1; only (1, 1) meets the SLA, exactly
    # (80 + 20 = 100 ms)
    b, v, t = B.best_batches(COST2, swap, 100.0, 1000.0, 4, pipelined=False)
    assert b == [1, 1] and t == 80.0


def test_no_feasible_choice():
    assert B.best_batches([[60.0, 70.0]], None, 100.0, 30.0, 2) is None


def _table(rng, n, nb):
    rows = []
    for _ in range(n):
        a = rng.uniform(1, 20)
        steps = [rng.uniform(0.2, 8) for _ in range(nb)]
        row, acc = [], a
        for s in steps:
            acc += s
            row.append(round(acc, 3))
        rows.append(row)
    return rows


@pytest.mark.parametrize("seed", range(12))
def test_monotone_in_sla_fps_and_swap(seed):
    rng = random.Random(seed)
    n, nb = rng.randint(2, 3), 5
    cost = _table(rng, n, nb)
    swap = [rng.uniform(0, 30) for _ in range(n)]
    fps = rng.choice([15.0, 30.0, 120.0])

    def val(sla, f=fps, s=swap):
        r = B.best_batches(cost, s, sla, f, nb)
        return -1.0 if r is None else r[1]
    for sla in (60.0, 100.0, 150.0):
        assert val(sla) <= val(sla + 50.0) + 1e-12
        assert val(sla, f=fps * 2) >= val(sla) - 1e-12
        assert val(sla, s=[0.0] * n) >= val(sla) - 1e-12
        r = B.best_batches(cost, swap, sla, fps, nb)
        if r is not None:
            assert B.feasible(cost, swap, r[0], sla)
            # no feasible list does better
            for b in [[rng.randint(1, nb) for _ in range(n)]
                      for _ in range(30)]:
                if B.feasible(cost, swap, b, sla):
                    assert B.min_throughput(cost, swap, b, fps) <= r[1] + 1e-12
