"""Round-robin schedules of model subsets for the weight-cache tests, sized
with the swap oracle (oracle/swap.py): the subsets follow the sharing-aware
load order, and the cache is a quarter larger than the most any round pins
(its own blobs and the next round's shared ones), grown until first-fit
placement runs the whole schedule."""

from __future__ import annotations

from dataclasses import dataclass


@dataclass
class Schedule:
    rounds: list        # model indices of each round
    order: list         # the oracle's load order
    sizes: list         # blob bytes
    users: list         # registered layers per blob
    per_model: list     # blobs of each model in first-use order
    need: int           # most bytes one round pins
    budget: int         # weight budget: cache plus resident scale/shift


def schedule(wl, per_round, cycles=2):
    from oracle import swap as S
    models = [(m.layers, m.in_chw) for m in wl.models]
    sizes, users, pm = S.blobs_of(models, wl.groups)
    order = S.load_order(sizes, pm, range(len(models)))
    cycle = [order[i:i + per_round] for i in range(0, len(order), per_round)]
    rounds = cycle * cycles

    def pinned(r):
        b = {x for m in rounds[r] for x in pm[m]}
        if r + 1 < len(rounds):
            b |= {x for m in rounds[r + 1] for x in pm[m] if users[x] > 1}
        return sum(sizes[x] for x in b)
    need = max(pinned(r) for r in range(len(rounds)))
    # scale/shift vectors stay resident: 2 x out_cp fp32 per blob, 256-byte
    # aligned
    aff = 0
    seen = set()
    for mi, (layers, chw) in enumerate(models):
        for li, l in enumerate(layers):
            key = next((tuple(g[0]) for g in wl.groups
                        if [mi, li] in [list(x) for x in g]), (mi, li))
            if l["op"] in ("conv", "fc") and key not in seen:
                seen.add(key)
                aff += (2 * ((l["cout"] + 7) // 8 * 8) * 4 + 255) // 256 * 256
    cap = need * 5 // 4 // 256 * 256
    while True:
        try:
            S.simulate(sizes, users, pm, cap, rounds)
            break
        except MemoryError:
            cap = cap * 5 // 4 // 256 * 256
    return Schedule(rounds, order, sizes, users, pm, need, aff + cap)
