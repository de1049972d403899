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

Parked keys and values live in pinned host memory mapped for the device, the
GPU&CPU hybrid storing of the paper's sec. 3: baton_kv_extract writes them
there and baton_kv_embed reads them back from there, each kernel moving the
tokens over the host link itself, with no device staging.  A return can also
be prefetched: prefetch() copies the next parked query's tokens to device
memory on a second stream while the step's attention runs, and grow() then
embeds from that copy once the copy's event has passed, so the return costs
the step a device-to-device embed instead of a transfer over the host link.
"""
import ctypes

from . import baton as B


def _cells(n_live, L):
    return n_live * L


_hip = None


def device_pointer(host_tensor):
    """The device address of a pinned host tensor (the HIP runtime's mapping)."""
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
    out = ctypes.c_void_p()
    rc = _hip.hipHostGetDevicePointer(ctypes.byref(out), ctypes.c_void_p(host_tensor.data_ptr()), ctypes.c_uint(0))
    if rc != 0 or not out.value:
        raise RuntimeError(f"hipHostGetDevicePointer failed ({rc}): the host buffer is not mapped for the device")
    return out.value


class BatchScaler:
    """Keeps live rows x padded length of `cache` (a BatonCache) at or below
    `max_cells`, parking queries in pinned host memory.  The cache's calls go
    to torch's current stream; prefetch copies go to a stream of their own
    (default priority) ordered against it by events."""

    def __init__(self, cache, max_cells):
        if max_cells < 1:
            raise ValueError("max_cells must be positive")
        self.cache = cache
        self.max_cells = max_cells
        # in the order they left: {"k", "v": pinned host tensors, "n": tokens,
        # "dk", "dv", "ready": a prefetched device copy and its event}
        self.parked = []
        self._side = None
        self._retiring = []   # host buffers a kernel may still read: (tensors, event)

    def footprint(self):
        L, _, lens = self.cache.query()
        return _cells(sum(1 for n in lens if n > 0), L)

    def _retire(self, tensors):
        """Keep host buffers alive until the current stream passes this point."""
        import torch
        ev = torch.cuda.Event()
        ev.record()
        self._retiring.append((tensors, ev))
        self._retiring = [(t, e) for t, e in self._retiring if not e.query()]

    def shrink(self):
        """Park queries until the footprint is within the threshold (one live
        query always stays).  Returns the slots vacated, in order."""
        moved = []
        while True:
            L, _, lens = self.cache.query()
            live = [b for b, n in enumerate(lens) if n > 0]
            if _cells(len(live), L) <= self.max_cells or len(live) <= 1:
                return moved

            def after(b):   # footprint without row b: release makes L the longest other span
                return _cells(len(live) - 1, max(lens[s] for s in live if s != b))
            b = min(live, key=lambda s: (after(s), -lens[s], s))
            self.parked.append(self._park(b))
            self.cache.evict([b], release=True)
            moved.append(b)

    def _park(self, b):
        """Slot b's keys and values into new pinned host buffers: the extract
        kernel writes them over the host link."""
        import torch
        n = self.cache.tokens()[b]
        shape = (self.cache.n_layers, self.cache.n_kv_heads, n, self.cache.head_dim)
        hk = torch.empty(shape, dtype=self.cache.k.dtype, pin_memory=True)
        hv = torch.empty(shape, dtype=self.cache.k.dtype, pin_memory=True)
        B.baton_kv_extract(self.cache.handle, [b], [device_pointer(hk)], [device_pointer(hv)],
                           torch.cuda.current_stream())
        return {"k": hk, "v": hv, "n": n, "dk": None, "dv": None, "ready": None}

    def prefetch(self):
        """Start copying the first parked query's keys and values to device
        memory on the prefetch stream (after everything the current stream has
        enqueued so far, so after its extract).  Returns whether a copy was
        started."""
        import torch
        if not self.parked or self.parked[0]["dk"] is not None:
            return False
        p = self.parked[0]
        if self._side is None:
            self._side = torch.cuda.Stream()   # default priority
        main = torch.cuda.current_stream()
        self._side.wait_stream(main)
        with torch.cuda.stream(self._side):
            p["dk"] = torch.empty(p["k"].shape, dtype=p["k"].dtype, device=self.cache.k.device)
            p["dv"] = torch.empty_like(p["dk"])
            p["dk"].copy_(p["k"], non_blocking=True)
            p["dv"].copy_(p["v"], non_blocking=True)
            p["ready"] = torch.cuda.Event()
            p["ready"].record(self._side)
        return True

    def grow(self):
        """Bring parked queries back, first parked first, into free slots while
        the footprint with them stays within the threshold.  A prefetched query
        is embedded from its device copy once the copy has passed; any other
        straight from pinned host memory.  Returns the slots they took, in
        order."""
        took = []
        while self.parked:
            L, _, lens = self.cache.query()
            free = [b for b, n in enumerate(lens) if n == 0]
            p = self.parked[0]
            n_live = sum(1 for n in lens if n > 0)
            if not free or _cells(n_live + 1, max(L, p["n"])) > self.max_cells:
                return took
            b = free[0]
            self._unpark(p, b)
            self.parked.pop(0)
            took.append(b)
        return took

    def _unpark(self, p, b):
        """A parked query into free slot b: from its prefetched device copy once
        the copy has passed, else straight from pinned host memory."""
        import torch
        stream = torch.cuda.current_stream()
        if p["dk"] is not None:
            stream.wait_event(p["ready"])
            self.cache.embed([b], [p["n"]], [p["dk"]], [p["dv"]])
            p["dk"].record_stream(stream)     # the allocator waits for the embed
            p["dv"].record_stream(stream)
        else:
            self.cache.embed([b], [p["n"]], [device_pointer(p["k"])], [device_pointer(p["v"])])
        self._retire((p["k"], p["v"]))
