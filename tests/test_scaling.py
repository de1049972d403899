"""The batch-size scaling policy's decisions (paper sec. 4.3), on the CPU: a
stand-in for the cache that keeps the handle's host metadata rules (end-aligned
rows, release to the longest live span on eviction, L = max(L, n) on embed,
+1 per step) and records the calls; the GPU lockstep test is
tests/test_gpu_preemption.py::test_batch_scaler_threshold."""
import torch

from paper_2410_18701_amd.scaling import BatchScaler


class Scaler(BatchScaler):
    """The policy with the data movement replaced by the stand-in's calls."""

    def _park(self, b):
        ks, _ = self.cache.extract([b])
        return {"n": ks[0].shape[2], "dk": None}

    def _unpark(self, p, b):
        t = torch.zeros((1, 1, p["n"], 8))
        self.cache.embed([b], [p["n"]], [t], [t.clone()])


class FakeCache:
    def __init__(self, batch, lens):
        self.lens = list(lens) + [0] * (batch - len(lens))
        self.L = max(self.lens)
        self.k = torch.empty(0)
        self.calls = []

    def query(self):
        return self.L, 0, list(self.lens)

    def extract(self, slots):
        (b,) = slots
        self.calls.append(("extract", b))
        t = torch.zeros((1, 1, self.lens[b], 8))
        return [t], [t.clone()]

    def tokens(self):
        return list(self.lens)

    def evict(self, slots, release=True):
        (b,) = slots
        self.calls.append(("evict", b))
        self.lens[b] = 0
        self.L = max(self.lens)

    def embed(self, slots, lens, ks, vs):
        (b,), (n,) = slots, lens
        assert self.lens[b] == 0 and ks[0].shape[2] == n
        self.calls.append(("embed", b, n))
        self.lens[b] = n
        self.L = max(self.L, n)

    def step(self):
        self.lens = [n + 1 if n else 0 for n in self.lens]
        self.L += 1


def test_longest_leaves_and_returns_when_it_fits():
    c = FakeCache(4, [36, 101, 26])
    s = Scaler(c, max_cells=300)
    assert s.footprint() == 303
    assert s.shrink() == [1]                       # 3 x 101 -> 2 x 36
    assert c.calls == [("extract", 1), ("evict", 1)] and s.footprint() == 72
    assert s.grow() == []                          # 3 x 101 with it back: refused
    c.evict([0])                                   # a query finishes: 1 x 26
    assert s.grow() == [0] and c.calls[-1] == ("embed", 0, 101)
    assert s.footprint() == 2 * 101 and not s.parked
    assert s.shrink() == []                        # a return never triggers a shrink


def test_shrink_stops_at_one_query_and_parks_in_order():
    c = FakeCache(4, [50, 60, 70, 80])
    s = Scaler(c, max_cells=40)
    assert s.shrink() == [3, 2, 1]                 # longest first; one query stays
    assert [p["n"] for p in s.parked] == [80, 70, 60]
    assert s.footprint() == 50
    c.evict([0])
    s.max_cells = 2 * 80
    assert s.grow() == [0, 1]                      # first parked first: 80, then 70 (2 x 80)
    assert [p["n"] for p in s.parked] == [60]      # 3 x 80 > 160: waits


def test_ties_go_to_the_longest_row():
    # two long rows: removing any one row leaves L at 100, so every removal
    # gives 2 x 100; the tie goes to the longest row (then the lowest slot)
    c = FakeCache(4, [100, 100, 10])
    s = Scaler(c, max_cells=250)
    assert s.shrink() == [0]                       # 3 x 100 -> 2 x 100 = 200
    assert s.footprint() == 200
