"""Batch-size scaling (paper sec. 4.3, "Batch size scaling"): the resources a
batch holds grow as its queries' keys and values grow, so they are watched
after each step; past a threshold some queries leave the batch for host
memory and their columns are released, and they come back, or new queries are
inserted, when the batch has room again.  Host logic over the C ABI: the moves
are baton_kv_extract / baton_kv_evict / baton_kv_embed.

The measure is the padded tensor the batch occupies in the paper's layout --
live rows x padded length L -- which is what overflows there.  A query that
leaves is the one whose removal shrinks that measure most (usually the
longest, which sets L); parked queries return in the order they left, each
only if the measure stays within the threshold with it back, so a returning
query never triggers the next shrink by itself.
"""


def _cells(n_live, L):
    return n_live * L


class BatchScaler:
    """Keeps live rows x padded length of `cache` (a BatonCache) at or below
    `max_cells`, parking queries in pinned host memory.  Everything is
    enqueued on torch's current stream, the copies to and from host memory
    included, so they stay ordered with the cache's own calls."""

    def __init__(self, cache, max_cells):
        if max_cells < 1:
            raise ValueError("max_cells must be positive")
        self.cache = cache
        self.max_cells = max_cells
        self.parked = []   # in the order they left: {"k", "v": pinned host tensors, "n": tokens}

    def footprint(self):
        L, _, lens = self.cache.query()
        return _cells(sum(1 for n in lens if n > 0), L)

    def shrink(self):
        """Park queries until the footprint is within the threshold (one live
        query always stays).  Returns the slots vacated, in order."""
        import torch
        moved = []
        while True:
            L, _, lens = self.cache.query()
            live = [b for b, n in enumerate(lens) if n > 0]
            if _cells(len(live), L) <= self.max_cells or len(live) <= 1:
                return moved

            def after(b):   # footprint without row b: release makes L the longest other span
                return _cells(len(live) - 1, max(lens[s] for s in live if s != b))
            b = min(live, key=lambda s: (after(s), -lens[s], s))
            ks, vs = self.cache.extract([b])
            pin = ks[0].is_cuda   # pinned host memory for device data
            hk = torch.empty(ks[0].shape, dtype=ks[0].dtype, pin_memory=pin)
            hv = torch.empty(vs[0].shape, dtype=vs[0].dtype, pin_memory=pin)
            hk.copy_(ks[0], non_blocking=True)
            hv.copy_(vs[0], non_blocking=True)
            self.cache.evict([b], release=True)
            self.parked.append({"k": hk, "v": hv, "n": ks[0].shape[2]})
            moved.append(b)

    def grow(self):
        """Bring parked queries back, first parked first, into free slots while
        the footprint with them stays within the threshold.  Returns the slots
        they took, in order."""
        took = []
        while self.parked:
            L, _, lens = self.cache.query()
            free = [b for b, n in enumerate(lens) if n == 0]
            p = self.parked[0]
            n_live = sum(1 for n in lens if n > 0)
            if not free or _cells(n_live + 1, max(L, p["n"])) > self.max_cells:
                return took
            b = free[0]
            dev = self.cache.k.device
            dk = p["k"].to(dev, non_blocking=True)
            dv = p["v"].to(dev, non_blocking=True)
            self.cache.embed([b], [p["n"]], [dk], [dv])
            self.parked.pop(0)
            took.append(b)
        return took
