"""Preemption and batch-size scaling on the GPU (sec. 4.3): a query's keys and
values stored aside with baton_kv_extract, the query evicted, other queries
taking and leaving its slot, and the stored query re-inserted later into a
different slot -- bit-exact against the oracle after every operation, and the
re-inserted query decoding as the oracle says it must."""
import numpy as np
import pytest
import torch

from paper_2410_18701_amd import baton as B
from paper_2410_18701_amd.cache import BatonCache
from tests import parity

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("shape", [("bf16", 2, 4, 8, 2, 128), ("f32", 1, 4, 4, 4, 64), ("bf16", 1, 5, 8, 8, 64)],
                         ids=lambda s: f"{s[0]}-{s[1]}x{s[2]}-{s[3]}/{s[4]}x{s[5]}")
def test_preempt_and_resume(shape):
    ops = [
        ("embed", [0, 1, 2], [37, 90, 12], [0, 1, 2]),
        ("step", 0), ("step", 1),
        ("extract", [1], "low"),                 # the lowest-priority query is stored aside
        ("evict", [1]),                          # ... and leaves its slot
        ("embed", [1], [50], [3]),               # the high-priority query takes it
        ("step", 2), ("step", 3),
        ("evict", [0]),                          # some query finishes
        ("embed_saved", [3], "low"),             # the stored one comes back, in another slot
        ("step", 4),
        ("extract", [3, 2], "pair"),             # batch-size scaling: two queries leave ...
        ("evict", [2, 3]),
        ("step", 5),
        ("embed_saved", [0, 2], "pair"),         # ... and return
        ("step", 6), ("step", 7),
    ]
    err = parity.run_script(shape, ops, capacity=256, split=64)
    print(f"[preempt] {shape}: max abs error {err:.3g}", flush=True)


def test_batch_scaler_threshold():
    """Batch-size scaling driven by a threshold (sec. 4.3): with live rows x
    padded length past it the query whose leaving shrinks that most -- the
    longest -- goes to pinned host memory and its columns are released; it
    stays parked while taking it back would pass the threshold again, and
    returns, into another slot, once a query has finished.  Bit-exact against
    the oracle after every operation, and the returned query decodes as the
    oracle says."""
    ops = [("embed", [0, 1, 2], [30, 95, 20], [0, 1, 2])]
    ops += [("step", s) for s in range(6)]        # L 101: 3 x 101 = 303 cells
    ops += [("scale", 300),                       # slot 1 (101 tokens) leaves: 2 x 36
            ("step", 6), ("step", 7),
            ("scale", 300),                       # 3 x 101 with it back: it stays out
            ("evict", [0]),                       # a query finishes: 1 x 28
            ("scale", 300),                       # 2 x 101: it returns, into slot 0
            ("step", 8), ("step", 9)]
    log = []
    err = parity.run_script(("bf16", 2, 4, 8, 2, 128), ops, capacity=256, split=64, log=log)
    assert log == [("scale", [1], []), ("scale", [], []), ("scale", [], [0])], log
    print(f"[scaler] {log}: max abs error {err:.3g}", flush=True)


def test_host_round_trip():
    """Batch-size scaling through host memory: extract, copy to pinned host
    memory, evict, copy back, re-embed -- the cache returns bit for bit."""
    cache = BatonCache(2, 3, 4, 2, 64, capacity=128, dtype="bf16")
    from workload import driver
    from workload.configs import Workload
    dev = driver.DeviceInputs(Workload("h", "bf16", 2, 3, 4, 2, 64, 1, 0, seed=4))
    srcs = [dev.prefill(q, n) for q, n in zip([0, 1, 2], [20, 33, 7])]
    cache.embed([0, 1, 2], [20, 33, 7], [s[0] for s in srcs], [s[1] for s in srcs])
    torch.cuda.synchronize()
    before = (parity.host_bits(cache.k).copy(), parity.host_bits(cache.v).copy(), cache.query())
    ks, vs = cache.extract([1])
    hk = torch.empty(ks[0].shape, dtype=ks[0].dtype, pin_memory=True)
    hv = torch.empty(vs[0].shape, dtype=vs[0].dtype, pin_memory=True)
    hk.copy_(ks[0])
    hv.copy_(vs[0])
    cache.evict([1], release=True)
    del ks, vs
    dk, dv = hk.cuda(), hv.cuda()
    cache.embed([1], [dk.shape[2]], [dk], [dv])
    torch.cuda.synchronize()
    assert cache.query() == before[2]
    assert np.array_equal(parity.host_bits(cache.k), before[0])
    assert np.array_equal(parity.host_bits(cache.v), before[1])
    with pytest.raises(B.BatonError) as e:
        cache.extract([2])[0]                     # live: fine
        B.baton_kv_extract(cache.handle, [1, 1], [dk, dk], [dv, dv])
    assert e.value.status == B.BATON_EINVAL
    cache.close()


def _device_pointer(host_ptr):
    """The device address of pinned host memory (HIP's own answer), or None."""
    import ctypes
    try:
        hip = ctypes.CDLL("libamdhip64.so")
    except OSError:
        return None
    out = ctypes.c_void_p()
    rc = hip.hipHostGetDevicePointer(ctypes.byref(out), ctypes.c_void_p(host_ptr), ctypes.c_uint(0))
    return out.value if rc == 0 else None


def test_direct_host_offload():
    """Batch-size scaling with the keys and values held in host memory: extract
    writes straight into pinned host buffers over PCIe, and embed reads them back
    from there, with no device staging -- the same bits as through device memory."""
    import time
    from workload import driver
    from workload.configs import Workload
    w = Workload("h", "bf16", 2, 4, 8, 2, 128, 1, 0, seed=5)
    dev = driver.DeviceInputs(w)
    lens = [40, 300, 17]
    caches = []
    for _ in range(2):
        c = BatonCache(2, 4, 8, 2, 128, capacity=512, dtype="bf16")
        srcs = [dev.prefill(q, n) for q, n in zip([0, 1, 2], lens)]
        c.embed([0, 1, 2], lens, [s[0] for s in srcs], [s[1] for s in srcs])
        caches.append(c)
    torch.cuda.synchronize()
    direct, staged = caches
    n = direct.tokens()[1]
    hk = torch.empty((2, 2, n, 128), dtype=torch.bfloat16, pin_memory=True)
    hv = torch.empty_like(hk, pin_memory=True)
    dk, dv = _device_pointer(hk.data_ptr()), _device_pointer(hv.data_ptr())
    if dk is None or dv is None:
        pytest.skip("pinned host memory is not mapped for the device")
    t0 = time.perf_counter()
    B.baton_kv_extract(direct.handle, [1], [dk], [dv], torch.cuda.current_stream())
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    print(f"[offload] {2 * hk.numel() * 2 / 1e6:.1f} MB extracted to host in {dt * 1e3:.2f} ms", flush=True)
    ks, vs = staged.extract([1])
    assert np.array_equal(parity.host_bits(ks[0]), hk.view(torch.int16).numpy().view(np.uint16))
    assert np.array_equal(parity.host_bits(vs[0]), hv.view(torch.int16).numpy().view(np.uint16))
    for c in caches:
        c.evict([1], release=True)
    B.baton_kv_embed(direct.handle, [3], [n], [dk], [dv], torch.cuda.current_stream())
    staged.embed([3], [n], ks, vs)
    for c in caches:
        c.flush()
    torch.cuda.synchronize()
    assert direct.query() == staged.query()
    assert np.array_equal(parity.host_bits(direct.k), parity.host_bits(staged.k))
    assert np.array_equal(parity.host_bits(direct.v), parity.host_bits(staged.v))
    for c in caches:
        c.close()


@pytest.mark.parametrize("shape", [("bf16", 2, 6, 8, 2, 128), ("f32", 1, 6, 4, 4, 64)],
                         ids=lambda s: f"{s[0]}-{s[1]}x{s[2]}-{s[3]}/{s[4]}x{s[5]}")
def test_move_and_compact(shape):
    """Queries moved between slots -- compaction of the live rows to the front,
    a move into a slot that still owes placeholders, a row with holes -- in
    lockstep with the oracle; later outputs as if they had always been there."""
    ops = [
        ("embed", [1, 3, 5], [30, 70, 12], [0, 1, 2]), ("step", 0),
        ("move", [3, 5], [0, 2]),                 # compact: live rows 0, 1, 2
        ("step", 1),
        ("evict", [1]), ("move", [2], [1]),       # the target owes the evicted query's tokens
        ("step", 2),
        ("shape", [2], [9], [3]), ("step", 3),    # a prefill step leaves holes in rows 0 and 1
        ("move", [0, 1], [4, 5]),                 # holey rows move
        ("step", 4), ("flush",), ("step", 5),
    ]
    err = parity.run_script(shape, ops, capacity=256, split=64)
    print(f"[move] {shape}: max abs error {err:.3g}", flush=True)


def test_batch_scaler_threshold_prefetched():
    """The same policy with the parked query's return prefetched to device
    memory on the scaler's second stream: the same decisions and the same
    bits as returning it straight from pinned host memory."""
    ops = [("embed", [0, 1, 2], [30, 95, 20], [0, 1, 2])]
    ops += [("step", s) for s in range(6)]
    ops += [("scale", 300, True), ("step", 6), ("step", 7), ("scale", 300, True), ("evict", [0]),
            ("scale", 300, True), ("step", 8), ("step", 9)]
    log = []
    err = parity.run_script(("bf16", 2, 4, 8, 2, 128), ops, capacity=256, split=64, log=log)
    assert log == [("scale", [1], []), ("scale", [], []), ("scale", [], [0])], log
    print(f"[scaler prefetched] {log}: max abs error {err:.3g}", flush=True)


def test_prefetched_return_overlaps_the_step():
    """A parked query's return over the host link: straight from pinned host
    memory after a step (the embed reads over the link on the step's stream)
    against prefetched to device memory on the second stream while the step's
    attention runs.  Both return the query's tokens bit for bit; the timings
    (HIP events on the step's stream) are printed."""
    from paper_2410_18701_amd.scaling import BatchScaler
    from workload import driver
    from workload.configs import Workload
    NL, Bt, Hq, Hkv, D, n = 8, 128, 64, 8, 128, 2000
    w = Workload("overlap", "bf16", NL, Bt, Hq, Hkv, D, n, 0, seed=6)
    w.init_lens = [n] * (Bt - 1) + [n // 2]
    cache, dev = driver.open_cache(w, capacity=n + 64)
    scaler = BatchScaler(cache, max_cells=10 ** 9)
    ins = [dev.decode(s, layer) for s in range(8) for layer in range(NL)]
    E = lambda: torch.cuda.Event(enable_timing=True)

    def step(s):
        for layer in range(NL):
            q, kn, vn = ins[s * NL + layer]
            cache.decode_attn(layer, q, kn, vn)
        cache.advance()

    step(0)
    torch.cuda.synchronize()
    a, b = E(), E()
    a.record()
    step(1)
    b.record()
    torch.cuda.synchronize()
    t_step = a.elapsed_time(b)
    times = {}
    # The first transfer on a new stream pays a one-time start-up (several ms
    # on a fresh process); the cycle "warmup" is not timed.
    for s, mode in ((2, "warmup"), (4, "direct"), (6, "prefetched")):
        L, _, lens = cache.query()
        victim = max((b for b in range(Bt) if lens[b] > 0), key=lambda b: (lens[b], -b))
        ks, vs = cache.extract([victim])              # the query before it leaves, to compare
        scaler.max_cells = (sum(1 for x in lens if x > 0) - 1) * L   # room for one row fewer
        parked = scaler.shrink()
        assert parked == [victim], (parked, victim)   # the longest rows tie; the lowest slot goes
        scaler.max_cells = 10 ** 9
        torch.cuda.synchronize()
        a, b = E(), E()
        a.record()
        if mode in ("prefetched", "warmup"):
            scaler.prefetch()
        step(s)
        back = scaler.grow()
        b.record()
        torch.cuda.synchronize()
        times[mode] = a.elapsed_time(b)
        assert len(back) == len(parked)
        slot = back[0]
        k2, v2 = cache.extract([slot])
        assert torch.equal(k2[0].view(torch.int16), ks[0].view(torch.int16))
        assert torch.equal(v2[0].view(torch.int16), vs[0].view(torch.int16))
        step(s + 1)
    mb = 2 * NL * Hkv * n * D * 2 / 1e6
    print(f"[overlap] step {t_step:.3f} ms; step + return of {mb:.0f} MB: straight from host memory "
          f"{times['direct']:.3f} ms, prefetched during the step {times['prefetched']:.3f} ms", flush=True)
    cache.close()
