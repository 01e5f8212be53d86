"""Oracle of the merging-aware swap schedule at the edge: rounds over subsets
of the registered models, a device weight cache kept across rounds, the
paper's eviction rule and a sharing-aware load order.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What the paper describes:
  - Section 3.2: when a workload's models do not all fit in GPU memory, the
    edge box time-shares them, visiting the models in round-robin order and
    swapping their weights in from CPU memory;
  - Section 5.4: with merging, loading the next model only has to bring in
    its layers that are not already in GPU memory, and models that share
    the most layers should be placed next to one another in the load order;
  - Appendix A.4: the scheduler keeps a list of the shared layers needed by
    the models currently in GPU memory or next in line to be loaded, and
    when it evicts, it evicts only weights of layers not in that list.

Readings taken here (the paper gives the policy, not its mechanics):
  - a blob is one stored parameter copy: one per merged group, one per
    unmerged conv / fc layer. Its cached bytes are its weights in kernel
    layout, [out_cp][k] with k = kh * kw * in_cp for a conv and
    H * W * C_p of the flattened producer for an fc (channel counts padded
    to multiples of 8), times the element size, rounded up to 256 bytes.
    Per-channel scale/shift vectors are always resident and not cached;
  - blobs are numbered by first appearance, models in id order and layers
    in layer order; a blob is shared when two or more registered layers
    use it;
  - the cache is `capacity` bytes; a blob is placed first-fit: at the lowest
    256-aligned offset whose free run is large enough;
  - round r runs the model set S_r and needs every blob of those models,
    taken in first-use order (models by id, then layers);
  - pinned during round r: every blob it needs, and every shared blob of the
    models of the next round (the models "next in line");
  - a needed blob not cached is loaded; while no free run fits it, one
    cached blob that is not pinned is evicted, chosen unshared before
    shared, then larger before smaller, then lower blob number; when none
    is left the round cannot run (its pinned blobs do not fit);
  - the round's loaded bytes are the cached bytes of the blobs it loaded;
  - load order of a round-robin cycle (one model per round): start with the
    model of the most blob bytes; then repeatedly place the remaining model
    that shares the most blob bytes with one end of the order so far, at
    that end (ties: more blob bytes, then lower index, then the back end),
    so that chains of sharing models are walked in both directions.
"""

from __future__ import annotations

ALIGN = 256


def _cp(c):
    return (c + 7) // 8 * 8


def blob_bytes(layers, in_chw, i, elem=2):
    """Cached bytes of layer i's parameter copy (conv or fc)."""
    from .merging import output_shapes
    shapes = output_shapes(layers, in_chw)
    l = layers[i]
    c, h, w = in_chw if l["src0"] < 0 else shapes[l["src0"]]
    if l["op"] == "conv":
        k = l["kh"] * l["kw"] * _cp(c)
    elif l["op"] == "fc":
        k = h * w * _cp(c)
    else:
        raise ValueError(l["op"])
    b = _cp(l["cout"]) * k * elem
    return (b + ALIGN - 1) // ALIGN * ALIGN


def blobs_of(models, groups, elem=2):
    """Blob table of registered models (list of (layers, in_chw), model id =
    index) under a sharing map (groups of (model, layer), first member the
    source): returns (sizes, users, per-model blob lists in first-use
    order)."""
    src = {}
    for g in groups:
        for mb in g:
            src[tuple(mb)] = tuple(g[0])
    number = {}
    sizes, users = [], []
    per_model = []
    for mi, (layers, in_chw) in enumerate(models):
        mine = []
        for li, l in enumerate(layers):
            if l["op"] not in ("conv", "fc"):
                continue
            key = src.get((mi, li), (mi, li))
            if key not in number:
                number[key] = len(sizes)
                sm, sl = key
                sizes.append(blob_bytes(models[sm][0], models[sm][1], sl, elem))
                users.append(0)
            b = number[key]
            users[b] += 1
            if b not in mine:
                mine.append(b)
        per_model.append(mine)
    return sizes, users, per_model


class Cache:
    """First-fit weight cache with the eviction rule above."""

    def __init__(self, capacity, sizes, users):
        self.capacity = capacity
        self.sizes = sizes
        self.shared = [u > 1 for u in users]
        self.at = {}          # blob -> offset

    def used(self):
        return sum(self.sizes[b] for b in self.at)

    def _hole(self, size):
        taken = sorted((o, o + self.sizes[b]) for b, o in self.at.items())
        pos = 0
        for lo, hi in taken:
            if lo - pos >= size:
                return pos
            pos = max(pos, hi)
        return pos if self.capacity - pos >= size else None

    def _victim(self, pinned):
        cands = [b for b in self.at if b not in pinned]
        if not cands:
            return None
        # unshared first, then larger, then lower number
        return min(cands, key=lambda b: (self.shared[b], -self.sizes[b], b))

    def run_round(self, needed, pinned):
        """Loads the needed blobs; returns (loaded, evicted) blob lists, or
        raises when the pinned blobs leave no room."""
        loaded, evicted = [], []
        for b in needed:
            if b in self.at:
                continue
            while True:
                off = self._hole(self.sizes[b])
                if off is not None:
                    break
                v = self._victim(pinned)
                if v is None:
                    raise MemoryError("pinned blobs do not leave room")
                del self.at[v]
                evicted.append(v)
            self.at[b] = off
            loaded.append(b)
        return loaded, evicted


def simulate(sizes, users, per_model, capacity, rounds):
    """Run the rounds (lists of model ids) through a cold cache; per round:
    (loaded bytes, evicted bytes, cached bytes after the round, loaded
    blobs, evicted blobs)."""
    cache = Cache(capacity, sizes, users)
    out = []
    n = len(rounds)
    for r, models in enumerate(rounds):
        needed = []
        for m in sorted(models):
            for b in per_model[m]:
                if b not in needed:
                    needed.append(b)
        pinned = set(needed)
        if r + 1 < n:
            for m in rounds[r + 1]:
                pinned.update(b for b in per_model[m] if users[b] > 1)
        loaded, evicted = cache.run_round(needed, pinned)
        out.append((sum(sizes[b] for b in loaded),
                    sum(sizes[b] for b in evicted), cache.used(),
                    loaded, evicted))
    return out


def shared_bytes(sizes, per_model, a, b):
    return sum(sizes[x] for x in set(per_model[a]) & set(per_model[b]))


def load_order(sizes, per_model, models):
    """Sharing-aware load order of `models` (model ids), as above."""
    left = list(models)
    total = {m: sum(sizes[b] for b in per_model[m]) for m in left}
    first = min(left, key=lambda m: (-total[m], m))
    order = [first]
    left.remove(first)
    while left:
        # (shared bytes with an end, more bytes, lower index, back end first)
        cands = [(-shared_bytes(sizes, per_model, order[end], m), -total[m],
                  m, 0 if end == -1 else 1)
                 for m in left for end in (-1, 0)]
        best = min(cands)
        m = best[2]
        if best[3] == 0:
            order.append(m)
        else:
            order.insert(0, m)
        left.remove(m)
    return order
