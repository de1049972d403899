"""GPU-vs-oracle parity harness.

Runs a workload's schedule through libbaton on the GPU and, step by step,
through the materialized CPU oracle fed from the host generator (same bits as
the device generator), comparing after every operation:
  * the K/V ring read off at the reported base: the first L columns must equal
    the oracle's aligned cache bit for bit, the other capacity - L columns must
    hold the placeholder;
  * the mask, bit for bit;
  * every layer's attention output, within the element type's tolerance.
"""
import math

import numpy as np
import torch

import oracle.baton_oracle as O
from workload import driver, gen

TOL = {"f32": 1e-5, "bf16": 2e-2}


def host_bits(t):
    """Device tensor -> numpy array of its stored bits."""
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    if t.dtype == torch.float32:
        return t.view(torch.int32).cpu().numpy().view(np.uint32)
    return t.cpu().numpy()


def ring_to_logical(ring, base, L):
    cap = ring.shape[3]
    idx = (np.arange(L) + base) % cap
    rest = (np.arange(L, cap) + base) % cap
    return ring[:, :, :, idx], ring[:, :, :, rest]


def check_ring(cache, pb, where):
    L, base, lens = cache.query()
    assert L == pb.L, (where, L, pb.L)
    assert lens == pb.lens, (where, lens, pb.lens)
    for which, want in (("k", pb.K), ("v", pb.V)):
        ring = host_bits(cache.k if which == "k" else cache.v)
        win, rest = ring_to_logical(ring, base, L)
        if not np.array_equal(win, want):
            bad = np.argwhere(win != want)
            raise AssertionError(f"{where}: {which} window differs at {len(bad)} positions, "
                                 f"first {bad[:5].tolist()}")
        assert np.all(rest == pb.fill), f"{where}: {which} unused ring columns are not placeholders"


def max_err(gpu_out, oracle_out, dtype):
    got = O.widen(host_bits(gpu_out), dtype)
    return float(np.max(np.abs(got - oracle_out))) if got.size else 0.0


def run(w, capacity=None, split=None, fill_bits=None, check_every_op=True, scale=0.0):
    """Drive the whole schedule; returns the largest attention error seen."""
    cache = driver.BatonCache(w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim,
                              w.capacity() if capacity is None else capacity, dtype=w.dtype,
                              fill_bits=fill_bits)
    if split is not None:
        cache.set_split_tokens(split)
    dev = driver.DeviceInputs(w)
    pb = O.PaddedBatch(w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.dtype,
                       fill_bits=cache.fill_bits)
    worst = 0.0

    def host_prefill(qid, n):
        return (gen.prefill_host(w.seed, "k", qid, w.n_layers, w.n_kv_heads, n, w.head_dim, w.dtype),
                gen.prefill_host(w.seed, "v", qid, w.n_layers, w.n_kv_heads, n, w.head_dim, w.dtype))

    def embed(slots, lens, qids):
        srcs = [dev.prefill(q, n) for q, n in zip(qids, lens)]
        cache.embed(slots, lens, [s[0] for s in srcs], [s[1] for s in srcs])
        hs = [host_prefill(q, n) for q, n in zip(qids, lens)]
        pb.embed(slots, lens, [h[0] for h in hs], [h[1] for h in hs])

    torch.cuda.synchronize()
    check_ring(cache, pb, "created")
    embed(list(range(w.batch)), w.init_lens, list(range(w.batch)))
    check_ring(cache, pb, "initial batch")
    sc = None if scale == 0.0 else scale
    for s, ev in enumerate(w.steps):
        cache.evict(ev.evict, release=True)
        pb.evict(ev.evict, release=True)
        if check_every_op:
            check_ring(cache, pb, f"step {s} evict")
        if ev.insert:
            embed(ev.insert, ev.insert_lens, ev.insert_qids)
            if check_every_op:
                check_ring(cache, pb, f"step {s} embed")
        m = cache.build_mask()
        assert np.array_equal(m.cpu().numpy(), pb.mask()), f"step {s} mask"
        for layer in range(w.n_layers):
            q, kn, vn = dev.decode(s, layer)
            out = cache.decode_attn(layer, q, kn, vn, scale=scale)
            hq = [gen.decode_host(w.seed, sid, s, layer, w.n_layers, w.batch, h, w.head_dim, w.dtype)
                  for sid, h in ((gen.S_Q, w.n_q_heads), (gen.S_KNEW, w.n_kv_heads),
                                 (gen.S_VNEW, w.n_kv_heads))]
            assert np.array_equal(host_bits(q), hq[0]), "device and host generators disagree"
            want = pb.decode_layer(layer, hq[0], hq[1], hq[2], scale=sc)
            err = max_err(out, want, w.dtype)
            worst = max(worst, err)
            assert err <= TOL[w.dtype], f"step {s} layer {layer}: max abs error {err}"
            free = [b for b in range(w.batch) if pb.lens[b] == 0]
            if free:
                assert np.all(host_bits(out)[free] == 0), "free rows must be exactly 0"
        cache.advance()
        pb.advance()
        if check_every_op or s == len(w.steps) - 1:
            check_ring(cache, pb, f"step {s} advance")
    cache.close()
    return worst
