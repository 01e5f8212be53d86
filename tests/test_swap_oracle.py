"""Pins of the swap-schedule oracle (oracle/swap.py) against closed forms,
constructed cases that separate each rule of the policy, invariants on
random instances, and brute force (Section 3.2 round-robin time sharing;
Section 5.4 loading only missing layers, sharing-aware load order;
Appendix A.4 pinning and eviction of unshared layers only)."""

import itertools
import random

import pytest

from oracle import swap as S


def _table(model_blobs, sizes):
    users = [0] * len(sizes)
    for bl in model_blobs:
        for b in bl:
            users[b] += 1
    return sizes, users, model_blobs


def test_blob_bytes_follow_the_kernel_layout():
    conv = dict(op="conv", src0=-1, cin=3, cout=64, kh=7, kw=7, stride=2,
                pad=3)
    # [64][7 * 7 * 8] bf16 = 50176 bytes, a multiple of 256
    assert S.blob_bytes([conv], (3, 224, 224), 0) == 64 * 49 * 8 * 2
    fc = dict(op="fc", src0=0, cin=64 * 112 * 112, cout=10)
    # out channels padded to 16, k = 112 * 112 * 64
    assert S.blob_bytes([conv, fc], (3, 224, 224), 1) == \
        16 * 112 * 112 * 64 * 2
    odd = dict(op="conv", src0=-1, cin=5, cout=3, kh=1, kw=1, stride=1,
               pad=0)
    assert S.blob_bytes([odd], (5, 4, 4), 0) == 256   # 8 * 8 * 2, aligned


def test_blob_table_counts_one_copy_per_group():
    from workloads import configs
    wl = configs.r50x2_vgg16x2(res=64, frames=1)
    models = [(m.layers, m.in_chw) for m in wl.models]
    sizes, users, per_model = S.blobs_of(models, wl.groups)
    merged = {tuple(g[0]) for g in wl.groups if len(g) > 1}
    param = sum(sum(1 for l in m.layers if l["op"] in ("conv", "fc"))
                for m in wl.models)
    # every parametric appearance is a blob, except merged members
    extra = sum(len(g) - 1 for g in wl.groups
                if wl.models[g[0][0]].layers[g[0][1]]["op"] in ("conv", "fc"))
    assert len(sizes) == param - extra
    assert sum(u > 1 for u in users) == sum(
        1 for g in wl.groups if len(g) > 1 and
        wl.models[g[0][0]].layers[g[0][1]]["op"] in ("conv", "fc"))
    assert merged  # the workload has merged layers
    # ResNet-50 b shares stem + layers 1-3 with a: its own blobs are layer4 + fc
    own_b = [b for b in per_model[1] if users[b] == 1]
    assert len(own_b) == sum(1 for l in wl.models[1].layers
                             if l["op"] in ("conv", "fc") and
                             (l["name"].startswith("layer4") or l["op"] == "fc"))


def test_everything_fits_loads_once():
    sizes, users, pm = _table([[0, 1], [1, 2], [3]], [512, 1024, 256, 768])
    rounds = [[0], [1], [2]] * 3
    out = S.simulate(sizes, users, pm, sum(sizes), rounds)
    assert [o[0] for o in out[:3]] == [1536, 256, 768]
    assert all(o[0] == 0 and o[1] == 0 for o in out[3:])


def test_disjoint_models_reload_everything_each_turn():
    # capacity of the largest model: every round evicts the other model
    sizes, users, pm = _table([[0, 1], [2, 3]], [1024, 512, 768, 768])
    out = S.simulate(sizes, users, pm, 1536, [[0], [1]] * 3)
    assert [o[0] for o in out] == [1536, 1536] * 3
    assert [o[1] for o in out] == [0, 1536, 1536, 1536, 1536, 1536]


def test_shared_layers_are_not_reloaded_between_neighbours():
    # blob 0 (1024 B) shared by both models; each has 512 B of its own
    sizes, users, pm = _table([[0, 1], [0, 2]], [1024, 512, 512])
    out = S.simulate(sizes, users, pm, 1536, [[0], [1]] * 3)
    assert [o[0] for o in out] == [1536] + [512] * 5
    assert all(0 in {b for b in range(3)} for _ in out)


def test_shared_layer_of_the_next_model_is_pinned():
    # blob 0 (1024 B) shared by models 1 and 2, blob 1 (512 B) shared by
    # models 2 and 3, blobs 2 and 3 model 0's own. Model 2 ran, model 0 runs
    # now and needs room for blob 3: the largest unpinned shared blob would
    # be blob 0, but with model 1 next it is pinned and blob 1 goes.
    sizes, users, pm = _table([[2, 3], [0], [0, 1], [1]], [1024, 512, 256, 512])
    for nxt, gone in (([1], [1]), ([], [0])):
        cache = S.Cache(1792, sizes, users)
        cache.run_round([0, 1], {0, 1})
        pinned = {2, 3} | {b for m in nxt for b in pm[m] if users[b] > 1}
        loaded, evicted = cache.run_round([2, 3], pinned)
        assert loaded == [2, 3] and evicted == gone, (nxt, evicted)


def test_unshared_blobs_are_evicted_before_shared_ones():
    # equal sizes: without the rule the lower number (the shared blob 0)
    # would go; the unshared blob 1 goes instead
    sizes, users, pm = _table([[0], [0], [1], [2]], [512, 512, 512])
    cache = S.Cache(1024, sizes, users)
    cache.run_round([0, 1], {0, 1})
    loaded, evicted = cache.run_round([2], {2})
    assert evicted == [1] and loaded == [2]
    # a larger blob needs both gone: unshared first, then shared
    sizes, users, pm = _table([[0], [0], [1], [2]], [512, 512, 768])
    cache = S.Cache(1024, sizes, users)
    cache.run_round([0, 1], {0, 1})
    loaded, evicted = cache.run_round([2], {2})
    assert evicted == [1, 0]


def test_first_fit_reuses_the_lowest_hole():
    sizes, users, pm = _table([[0], [1], [2], [3]], [512, 256, 512, 256])
    cache = S.Cache(1280, sizes, users)
    cache.run_round([0, 1, 2], {0, 1, 2})
    assert cache.at == {0: 0, 1: 512, 2: 768}
    # blob 3 (256 B) fits the tail? 1280 - 1280 = 0: evict (largest first,
    # lowest number on ties: blob 0), then first fit at offset 0
    loaded, evicted = cache.run_round([3], {3})
    assert evicted == [0] and cache.at[3] == 0


def test_pinned_blobs_that_do_not_fit_raise():
    sizes, users, pm = _table([[0, 1]], [1024, 1024])
    with pytest.raises(MemoryError):
        S.simulate(sizes, users, pm, 1536, [[0]])


def _random_case(rng, n_models=5, n_blobs=12):
    sizes = [rng.choice([256, 512, 768, 1024, 2048]) for _ in range(n_blobs)]
    pm = []
    for _ in range(n_models):
        k = rng.randint(1, 5)
        pm.append(sorted(rng.sample(range(n_blobs), k)))
    return _table(pm, sizes)


@pytest.mark.parametrize("seed", range(40))
def test_invariants_on_random_schedules(seed):
    rng = random.Random(seed)
    sizes, users, pm = _random_case(rng)
    need = max(sum(sizes[b] for b in bl) for bl in pm)
    # next round's shared blobs are pinned too: enough room for both
    cap = need + max(sum(sizes[b] for b in bl) for bl in pm) + rng.choice(
        [0, 256, 1024, 4096])
    rounds = [[rng.randrange(len(pm))] for _ in range(12)]
    cache = S.Cache(cap, sizes, users)
    prev = set()
    for r, models in enumerate(rounds):
        needed = []
        for m in sorted(models):
            needed += [b for b in pm[m] if b not in needed]
        pinned = set(needed)
        if r + 1 < len(rounds):
            pinned |= {b for m in rounds[r + 1] for b in pm[m] if users[b] > 1}
        before = set(cache.at)
        loaded, evicted = cache.run_round(needed, pinned)
        # loads exactly the needed blobs that were missing, in order
        assert loaded == [b for b in needed if b not in before]
        assert not (set(evicted) & pinned)
        assert set(needed) <= set(cache.at)
        assert cache.used() <= cap
        # placements are disjoint and inside the cache
        spans = sorted((o, o + sizes[b]) for b, o in cache.at.items())
        for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
            assert a1 <= b0
        assert all(o % 256 == 0 and o + sizes[b] <= cap
                   for b, o in cache.at.items())
        prev = set(cache.at)
    assert prev


def _cycle_shared(sizes, pm, order):
    return sum(S.shared_bytes(sizes, pm, a, b)
               for a, b in zip(order, order[1:]))


@pytest.mark.parametrize("seed", range(10))
def test_load_order_finds_chains(seed):
    """Models that share along a chain (each with its neighbours only, the
    shared blobs growing along it): the greedy order walks the chain, the
    order brute force finds to maximise the bytes shared by neighbours."""
    rng = random.Random(seed)
    n = rng.randint(3, 6)
    sizes, pm = [], [[] for _ in range(n)]
    perm = list(range(n))
    rng.shuffle(perm)
    for k in range(n - 1):   # shared blob between chain positions k, k+1
        sizes.append(256 * (k + 2))
        pm[perm[k]].append(len(sizes) - 1)
        pm[perm[k + 1]].append(len(sizes) - 1)
    for m in range(n):       # a small private blob each
        sizes.append(256)
        pm[m].append(len(sizes) - 1)
    sizes, users, pm = _table([sorted(x) for x in pm], sizes)
    order = S.load_order(sizes, pm, range(n))
    assert sorted(order) == list(range(n))
    best = max(_cycle_shared(sizes, pm, list(p))
               for p in itertools.permutations(range(n)))
    assert _cycle_shared(sizes, pm, order) == best


@pytest.mark.parametrize("seed", range(10))
def test_load_order_starts_from_the_largest_model(seed):
    """The order is a permutation in which the model of the most blob bytes
    sits next to a model that shares the most bytes with it (the first
    step of the greedy)."""
    rng = random.Random(100 + seed)
    sizes, users, pm = _random_case(rng, n_models=6)
    order = S.load_order(sizes, pm, range(6))
    assert sorted(order) == list(range(6))
    tot = [sum(sizes[b] for b in bl) for bl in pm]
    big = min(range(6), key=lambda m: (-tot[m], m))
    i = order.index(big)
    neigh = [order[j] for j in (i - 1, i + 1) if 0 <= j < 6]
    best = max(S.shared_bytes(sizes, pm, big, m) for m in range(6) if m != big)
    assert any(S.shared_bytes(sizes, pm, big, n) == best for n in neigh)
