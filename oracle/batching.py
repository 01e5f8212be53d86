"""Oracle of the SLA batch-size choice of a round-robin schedule.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What the paper describes (Section 3.2, the time-sharing variant of Nexus it
evaluates against and that the edge box runs before merging pays off, and
Section 5.4, where merging changes the swap delays the profiling uses):
models are visited in a round-robin order; an offline profiling pass picks
one global list of per-model batch sizes, the one that maximises the
minimum per-model throughput while every frame meets a processing
deadline (the SLA; 100 ms in the paper's experiments, Section 6.1); loading
the next model is pipelined with the current model's inference.

Readings taken here (the paper names the objective, not the arithmetic):
  - cost[m][b - 1] is model m's inference time for a batch of b frames,
    swap[m] the time to load what model m needs when its turn comes (0
    when everything is resident), both in ms;
  - one cycle visits every model once in the given order. Pipelined, the
    load of the next model overlaps the current model's inference, so a
    visit takes max(cost of the current batch, swap of the next model) and
    the cycle T = sum over i of max(cost[o_i](b), swap[o_(i+1)]) (cyclic);
    not pipelined, T = sum over m of (swap[m] + cost[m](b_m));
  - a frame that arrives just after its model's batch was formed waits one
    cycle and is then processed in the next batch: its latency is at most
    T + cost[m](b_m), which must not exceed the SLA for every model;
  - model m then processes b_m frames per cycle, min(b_m / T, fps) frames
    per second (it cannot process more frames than arrive);
  - the choice maximises the minimum of these over the models; ties are
    broken by the shorter cycle, then by the lexicographically smaller
    batch list. Batches range over 1..max_batch.

The oracle is brute force over every batch list: the definition written
out, for the small cases the tests use.
"""

from __future__ import annotations

import itertools


def cycle_ms(cost, swap, b, pipelined=True):
    """Cycle time T (ms) of batch list b (one entry per model, >= 1)."""
    n = len(b)
    c = [cost[m][b[m] - 1] for m in range(n)]
    s = list(swap) if swap is not None else [0.0] * n
    if pipelined:
        return sum(max(c[i], s[(i + 1) % n]) for i in range(n))
    return sum(s[m] + c[m] for m in range(n))


def feasible(cost, swap, b, sla_ms, pipelined=True):
    t = cycle_ms(cost, swap, b, pipelined)
    return all(t + cost[m][b[m] - 1] <= sla_ms for m in range(len(b)))


def min_throughput(cost, swap, b, fps, pipelined=True):
    """Minimum over the models of min(b_m / T, fps), in frames/s."""
    t = cycle_ms(cost, swap, b, pipelined) / 1000.0
    return min(min(x / t, fps) for x in b)


def best_batches(cost, swap, sla_ms, fps, max_batch, pipelined=True):
    """(batch list, min throughput, cycle ms) of the best feasible choice,
    or None when even batches of one frame miss the SLA."""
    n = len(cost)
    best = None
    for b in itertools.product(range(1, max_batch + 1), repeat=n):
        if not feasible(cost, swap, b, sla_ms, pipelined):
            continue
        v = min_throughput(cost, swap, b, fps, pipelined)
        t = cycle_ms(cost, swap, b, pipelined)
        key = (-v, t, b)
        if best is None or key < best[0]:
            best = (key, list(b), v, t)
    if best is None:
        return None
    return best[1], best[2], best[3]
