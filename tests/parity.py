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
import json
import math
import os

import numpy as np
import torch

import oracle.baton_oracle as O
from workload import driver, gen

TOL = {"f32": 1e-5, "bf16": 2e-2}

# Largest attention error of each parity run, by test: written at the end of
# the session (tests/conftest.py) so that the margins to the tolerances are kept.
MARGINS = []


def note_margin(worst, dtype, what=""):
    test = os.environ.get("PYTEST_CURRENT_TEST", "").split(" (")[0]
    MARGINS.append({"test": test, "what": what, "dtype": dtype, "max_abs_err": float(worst),
                    "tol": TOL[dtype], "frac_of_tol": round(float(worst) / TOL[dtype], 4)})


def write_margins(path):
    """Adds this session's margins to those already in the file."""
    if not MARGINS:
        return
    os.makedirs(os.path.dirname(path), exist_ok=True)
    old = []
    if os.path.exists(path):
        try:
            with open(path) as f:
                old = json.load(f)
        except (OSError, ValueError):
            old = []
    with open(path, "w") as f:
        json.dump(old + MARGINS, f, indent=1)


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


def check_ring(cache, pb, where, live_only=False, tokens_only=False):
    """live_only: compare the live rows' windows only (between an eviction and
    the next step, evicted rows may still hold their old tokens).  tokens_only:
    compare the live rows' tokens only, the columns the oracle's mask holds 1
    on (after an eviction without scrubbing, every other position may hold
    stale bytes)."""
    L, base, lens = cache.query()
    assert L == pb.L, (where, L, pb.L)
    assert lens == pb.lens, (where, lens, pb.lens)
    live = [b for b in range(len(lens)) if lens[b] > 0]
    for which, want in (("k", pb.K), ("v", pb.V)):
        ring = host_bits(cache.k if which == "k" else cache.v)
        win, rest = ring_to_logical(ring, base, L)
        if tokens_only:
            for b in live:
                cols = np.flatnonzero(pb.M[b, :L])
                if not np.array_equal(win[:, b][:, :, cols], want[:, b][:, :, cols]):
                    raise AssertionError(f"{where}: {which} tokens of slot {b} differ")
            continue
        if live_only:
            win, want = win[:, live], want[:, live]
        if not np.array_equal(win, want):
            bad = np.argwhere(win != want)
            raise AssertionError(f"{where}: {which} window differs at {len(bad)} positions, "
                                 f"first {bad[:5].tolist()}")
        if not live_only:
            assert np.all(rest == pb.fill), f"{where}: {which} unused ring columns are not placeholders"


def max_err(gpu_out, oracle_out, dtype):
    got = O.widen(host_bits(gpu_out), dtype)
    return float(np.max(np.abs(got - oracle_out))) if got.size else 0.0


def padded_kv(n_layers, batch, n_kv_heads, capacity, head_dim, dtype, pad=4096 + 16):
    """K and V as [n_layers][batch][n_kv_heads][capacity][head_dim] views of two
    buffers whose layers are `pad` elements longer than their rows (a layer
    stride the library is told, not a packed one); the padding is filled with
    a marker that the tests check is never written."""
    per = batch * n_kv_heads * capacity * head_dim
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    bufs = [torch.full((n_layers, per + pad), 7.0, dtype=tdt, device="cuda") for _ in range(2)]
    views = [b[:, :per].view(n_layers, batch, n_kv_heads, capacity, head_dim) for b in bufs]
    return views[0], views[1], lambda: all(bool((b[:, per:] == 7.0).all()) for b in bufs)


def run(w, capacity=None, split=None, fill_bits=None, check_every_op=True, scale=0.0, layout="by_layer",
        release_every=1, scrub=True):
    """Drive the whole schedule; returns the largest attention error seen.

    release_every: step s's evictions release (BATON_RELEASE) only when
    s % release_every == release_every - 1, and a release of no slot closes
    the run when release_every > 1.  scrub: evictions overwrite the finished
    queries' tokens with placeholders (BATON_SCRUB); without it, once a query
    has been evicted, only the live rows' tokens are compared."""
    cap = w.capacity() if capacity is None else capacity
    if layout == "padded":
        # two allocations whose layers are 4096 + 16 elements apart beyond their rows
        k, v, padding_intact = padded_kv(w.n_layers, w.batch, w.n_kv_heads, cap, w.head_dim, w.dtype)
        cache = driver.BatonCache(w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, cap,
                                  dtype=w.dtype, fill_bits=fill_bits, k=k, v=v)
    else:
        cache = driver.BatonCache(w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, cap,
                                  dtype=w.dtype, fill_bits=fill_bits, layout=layout)
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
    stale = False   # some eviction left its tokens in place
    for s, ev in enumerate(w.steps):
        release = s % release_every == release_every - 1
        cache.evict(ev.evict, release=release, scrub=scrub)
        pb.evict(ev.evict, release=release)
        stale |= bool(ev.evict) and not scrub
        if check_every_op:
            check_ring(cache, pb, f"step {s} evict", live_only=True, tokens_only=stale)
        if ev.insert:
            embed(ev.insert, ev.insert_lens, ev.insert_qids)
            if check_every_op:
                check_ring(cache, pb, f"step {s} embed", live_only=True, tokens_only=stale)
        if check_every_op and s % 2 == 1:
            cache.flush()
            torch.cuda.synchronize()
            check_ring(cache, pb, f"step {s} flush", tokens_only=stale)
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
            check_ring(cache, pb, f"step {s} advance", tokens_only=stale)
    if release_every > 1:
        cache.evict([], release=True, scrub=scrub)
        pb.evict([], release=True)
        torch.cuda.synchronize()
        check_ring(cache, pb, "closing release", tokens_only=stale)
    if layout == "padded":
        torch.cuda.synchronize()
        assert padding_intact(), "a write landed in the padding between layers"
    cache.close()
    note_margin(worst, w.dtype, w.name)
    return worst


# ------------------------------------------------------------ sampled mode --
class History:
    """Where each slot's query came from, to rebuild any row's history on the host.

    wide_steps: steps that prefilled new queries inside the batch; a live row's
    token of such a step is position 0 of that step's wide inputs."""

    def __init__(self, w, wide_steps=()):
        self.w = w
        self.qid = list(range(w.batch))
        self.plen = list(w.init_lens)
        self.first_step = [0] * w.batch      # first decode step of the query
        self.wide_steps = set(wide_steps)

    def insert(self, slot, qid, n, step):
        self.qid[slot], self.plen[slot], self.first_step[slot] = qid, n, step

    def row(self, slot, layer, head, step, which):
        """Host bits [n, D] of the query's own K (which='k') or V tokens for layer/head,
        including the token decoded at `step`."""
        w = self.w
        sid = gen.S_PREFILL_K if which == "k" else gen.S_PREFILL_V
        c0, st = gen.prefill_counter(self.qid[slot], w.n_layers, w.n_kv_heads, w.head_dim,
                                     layer0=layer, head0=head)
        pre = gen.fill_host(w.seed, sid, w.dtype, (1, 1, self.plen[slot], w.head_dim), c0, st)[0, 0]
        toks = []
        for s in range(self.first_step[slot], step + 1):
            if s in self.wide_steps:
                dsid = gen.S_KW if which == "k" else gen.S_VW
                c0, st = gen.wide_counter(s, layer, w.n_layers, w.batch, w.n_kv_heads, w.head_dim)
                c0 += slot * st[0] + head * w.head_dim       # position 0 of the slot
            else:
                dsid = gen.S_KNEW if which == "k" else gen.S_VNEW
                c0, st = gen.decode_counter(s, layer, w.n_layers, w.batch, w.n_kv_heads, w.head_dim)
                c0 += (slot * w.n_kv_heads + head) * w.head_dim
            toks.append(gen.fill_host(w.seed, dsid, w.dtype, (1, 1, 1, w.head_dim), c0, st)[0, 0])
        return np.concatenate([pre] + toks) if toks else pre


def check_placeholders_outside_live(cache, fill_bits, mask=None):
    """On the GPU: a ring position holds non-placeholder bits iff it is a live
    token (per the contiguous lengths, or the given 0-1 mask [B][>= L] of the
    cached columns when rows have holes)."""
    L, base, lens = cache.query()
    cap = cache.capacity
    col = torch.arange(cap, device=cache.k.device)
    logical = (col - base) % cap                                 # logical column of each physical one
    if mask is None:
        lens_t = torch.tensor(lens, device=cache.k.device)[:, None]
        live = (logical[None, :] < L) & (logical[None, :] >= L - lens_t) & (lens_t > 0)   # [B][cap]
    else:
        m = torch.zeros((cache.batch, cap + 1), dtype=torch.bool, device=cache.k.device)
        m[:, :L] = mask[:, :L].bool()
        live = m[:, torch.where(logical < L, logical, cap)]
    if cache.k.dtype == torch.bfloat16:
        idt, fill = torch.int16, int(np.array(fill_bits, np.uint16).view(np.int16))
    else:
        idt, fill = torch.int32, int(np.array(fill_bits, np.uint32).view(np.int32))
    for buf in (cache.k, cache.v):
        for layer in range(buf.shape[0]):
            for b0 in range(0, cache.batch, 16):
                rows = buf[layer, b0:b0 + 16].view(idt)
                written = (rows != fill).any(dim=-1)                            # [b][H][cap]
                want = live[b0:b0 + 16, None, :].expand_as(written)
                if not torch.equal(written, want):
                    raise AssertionError(f"layer {layer} rows {b0}..: placeholders and live tokens disagree")


def run_sampled(w, sample_steps, sample_layers, n_slots=4, seed=0, split=None, capacity=None):
    """Whole schedule on the GPU; the oracle checks metadata at every step and,
    at the sampled (step, layer) points, whole rows of K/V (bit-exact) and the
    attention output of every q-head of the sampled slots."""
    rng = np.random.default_rng(seed)
    cache, dev = driver.open_cache(w, capacity=capacity, split=split)
    pb = O.PaddedBatch(w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.dtype,
                       fill_bits=cache.fill_bits, materialize=False)
    pb.embed(list(range(w.batch)), w.init_lens, [None] * w.batch, [None] * w.batch)
    hist = History(w)
    g = w.n_q_heads // w.n_kv_heads
    worst, checked = 0.0, 0
    for s, ev in enumerate(w.steps):
        cache.evict(ev.evict, release=True)
        pb.evict(ev.evict, release=True)
        if ev.insert:
            srcs = [dev.prefill(q, n) for q, n in zip(ev.insert_qids, ev.insert_lens)]
            cache.embed(ev.insert, ev.insert_lens, [x[0] for x in srcs], [x[1] for x in srcs])
            pb.embed(ev.insert, ev.insert_lens, [None] * len(ev.insert), [None] * len(ev.insert))
            for slot, q, n in zip(ev.insert, ev.insert_qids, ev.insert_lens):
                hist.insert(slot, q, n, s)
            del srcs
        L, base, lens = cache.query()
        assert (L, lens) == (pb.L, pb.lens), f"step {s}: metadata"
        if s in sample_steps:
            m = cache.build_mask().cpu().numpy()
            assert np.array_equal(m, O.build_mask(pb.L, pb.lens)), f"step {s}: mask"
        live = pb.live()
        for layer in range(w.n_layers):
            q, kn, vn = dev.decode(s, layer)
            out = cache.decode_attn(layer, q, kn, vn)
            if s not in sample_steps or layer not in sample_layers:
                continue
            slots = sorted(set(rng.choice(live, min(n_slots, len(live)), replace=False).tolist())
                           | set(x for x in ev.insert if x in live))
            qh = host_bits(q)
            oh = O.widen(host_bits(out), w.dtype)
            for b in slots:
                for h in range(w.n_kv_heads):
                    kh = hist.row(b, layer, h, s, "k")
                    vh = hist.row(b, layer, h, s, "v")
                    assert len(kh) == pb.lens[b] + 1
                    # cached columns (before this step's token) of the ring, bit for bit
                    cols = (np.arange(pb.L - pb.lens[b], pb.L) + base) % cache.capacity
                    ring_k = host_bits(cache.k[layer, b, h, torch.as_tensor(cols, device=cache.k.device)])
                    ring_v = host_bits(cache.v[layer, b, h, torch.as_tensor(cols, device=cache.k.device)])
                    assert np.array_equal(ring_k, kh[:-1]) and np.array_equal(ring_v, vh[:-1]), \
                        f"step {s} layer {layer} slot {b} head {h}: cached tokens"
                    K, V = O.widen(kh, w.dtype), O.widen(vh, w.dtype)
                    for gi in range(g):
                        hq = h * g + gi
                        want = O.attend(O.widen(qh[b, hq], w.dtype), K, V, 1.0 / math.sqrt(w.head_dim))
                        err = float(np.max(np.abs(oh[b, hq] - want)))
                        worst = max(worst, err)
                        checked += 1
                        assert err <= TOL[w.dtype], f"step {s} layer {layer} slot {b} q-head {hq}: {err}"
            free = [b for b in range(w.batch) if pb.lens[b] == 0]
            if free:
                assert np.all(host_bits(out)[free] == 0)
        cache.advance()
        for layer in range(w.n_layers):
            pb.decode_layer(layer, None, None, None)
        pb.advance()
    torch.cuda.synchronize()
    check_placeholders_outside_live(cache, cache.fill_bits)
    cache.close()
    note_margin(worst, w.dtype, f"{w.name} sampled")
    return worst, checked


def run_sampled_no_pd(w, sample_steps, sample_layers=(0,), n_slots=4, n_pos=6, heads=(0,), seed=0):
    """The schedule without prefill/decode separation, whole on the GPU (the
    bench's launch configuration); metadata and the mask's width at every step;
    at the sampled steps the whole mask, and for sampled rows their K/V at the
    mask's ones (bit for bit, holes skipped) and outputs: a live row's position
    0 over its history, a new query's sampled positions causally over its prompt."""
    rng = np.random.default_rng(seed)
    wide = [s for s, ev in enumerate(w.steps) if ev.insert]
    cache, dev = driver.open_cache(w, no_pd=True)
    pb = O.PaddedBatch(w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.dtype,
                       fill_bits=cache.fill_bits, materialize=False)
    pb.embed(list(range(w.batch)), w.init_lens, [None] * w.batch, [None] * w.batch)
    hist = History(w, wide)
    g = w.n_q_heads // w.n_kv_heads
    sc = 1.0 / math.sqrt(w.head_dim)
    worst, checked = 0.0, 0
    for s, ev in enumerate(w.steps):
        cache.evict(ev.evict, release=True)
        pb.evict(ev.evict, release=True)
        ins = list(zip(ev.insert, ev.insert_qids, ev.insert_lens))
        if ins:
            cache.shape_insert(ev.insert, ev.insert_lens)
            pb.shape_insert(ev.insert, ev.insert_lens)
        T = pb.step_width()
        L, base, lens = cache.query()
        assert (L, lens) == (pb.L, pb.lens), f"step {s}: metadata"
        m = cache.build_mask()
        assert m.shape[1] == L + T
        M = pb.mask()
        if s in sample_steps:
            assert np.array_equal(m.cpu().numpy(), M), f"step {s}: mask"
        live = pb.live()
        for layer in range(w.n_layers):
            q, kn, vn = dev.prefill_step(s, layer, T, ins) if ins else dev.decode(s, layer)
            out = cache.decode_attn(layer, q, kn, vn)
            if s not in sample_steps or layer not in sample_layers:
                continue
            qh = host_bits(q) if ins else host_bits(q)[:, None]
            oh = O.widen(host_bits(out), w.dtype) if ins else O.widen(host_bits(out), w.dtype)[:, None]
            rows = sorted(set(rng.choice(live, min(n_slots, len(live)), replace=False).tolist()))
            for b in rows:
                keep = np.flatnonzero(M[b, :L])
                cols = torch.as_tensor((keep + base) % cache.capacity, device=cache.k.device)
                for h in heads:
                    kh = hist.row(b, layer, h, s, "k")
                    vh = hist.row(b, layer, h, s, "v")
                    assert len(kh) == len(keep) + 1, (s, b, len(kh), len(keep))
                    assert np.array_equal(host_bits(cache.k[layer, b, h, cols]), kh[:-1]) and \
                        np.array_equal(host_bits(cache.v[layer, b, h, cols]), vh[:-1]), \
                        f"step {s} layer {layer} slot {b} head {h}: cached tokens"
                    K, V = O.widen(kh, w.dtype), O.widen(vh, w.dtype)
                    for hq in range(h * g, h * g + g):
                        want = O.attend(O.widen(qh[b, 0, hq], w.dtype), K, V, sc)
                        err = float(np.max(np.abs(oh[b, 0, hq] - want)))
                        worst, checked = max(worst, err), checked + 1
                        assert err <= TOL[w.dtype], f"step {s} slot {b} q-head {hq}: {err}"
            for b, qid, p in ins:
                pos = sorted(set([0, p - 1] + rng.integers(0, p, size=n_pos).tolist()))
                for h in heads:
                    c0, st = gen.prompt_counter(qid, layer, w.n_layers, w.n_kv_heads, w.head_dim)
                    Kp = gen.fill_host(w.seed, gen.S_PREFILL_K, w.dtype, (1, p, w.n_kv_heads, w.head_dim), c0, st)[0, :, h]
                    Vp = gen.fill_host(w.seed, gen.S_PREFILL_V, w.dtype, (1, p, w.n_kv_heads, w.head_dim), c0, st)[0, :, h]
                    K, V = O.widen(Kp, w.dtype), O.widen(Vp, w.dtype)
                    for hq in range(h * g, h * g + g):
                        for i in pos:
                            t = T - p + i
                            want = O.attend(O.widen(qh[b, t, hq], w.dtype), K[:i + 1], V[:i + 1], sc)
                            err = float(np.max(np.abs(oh[b, t, hq] - want)))
                            worst, checked = max(worst, err), checked + 1
                            assert err <= TOL[w.dtype], f"step {s} new slot {b} pos {i} q-head {hq}: {err}"
        cache.advance()
        for layer in range(w.n_layers):
            pb.decode_layer(layer, None, None, None)
        pb.advance()
        for b, qid, p in ins:
            hist.insert(b, qid, p, s + 1)
    torch.cuda.synchronize()
    cache.flush()
    check_placeholders_outside_live(cache, cache.fill_bits, mask=cache.build_mask())
    cache.close()
    note_margin(worst, w.dtype, f"{w.name} sampled, no P&D")
    return worst, checked


# ---------------------------------------------------------- scripted mode --
def run_script(shape, ops, seed=3, capacity=64, split=None, layout="by_layer", log=None, scale=0.0):
    """A scripted sequence on a small batch, GPU and materialized oracle in
    lockstep, everything compared after every operation.

    shape: (dtype, n_layers, batch, n_q_heads, n_kv_heads, head_dim).  ops:
      ("embed", slots, lens, qids)   prefilled queries from the generator
      ("evict", slots)               with release and scrub
      ("evict", slots, release, scrub)  with the given flags
      ("extract", slots, tag)        store the slots' K/V aside (GPU and oracle)
      ("embed_saved", slots, tag)    re-insert stored queries into these slots
      ("shape", slots, lens, qids)   prefill new queries inside the batch in the next step
      ("move", src, dst)             live queries change slots
      ("step", s)                    mask, every layer with step-s inputs, advance
      ("flush",)                     the placeholder writes evictions still owe
      ("scale", max_cells)           BatchScaler.shrink then grow at this threshold (the
                                     oracle repeats its parks and returns; `log` gets
                                     ("scale", parked slots, returned slots))
      ("scale", max_cells, True)     the same with the return prefetched to device memory
                                     on the scaler's second stream first
    After a step or a flush the whole ring is compared; after the other
    operations the live rows (evicted rows may still hold old tokens); once an
    eviction did not scrub, the live rows' tokens only.  scale: the attention
    scale passed to every decode_attn (0: 1/sqrt(head_dim)).
    """
    dtype, NL, B, Hq, Hkv, D = shape
    from workload.configs import Workload
    w = Workload("script", dtype, NL, B, Hq, Hkv, D, 1, 0, seed=seed)
    cache = driver.BatonCache(NL, B, Hq, Hkv, D, capacity, dtype=dtype, layout=layout)
    if split is not None:
        cache.set_split_tokens(split)
    dev = driver.DeviceInputs(w)
    pb = O.PaddedBatch(NL, B, Hq, Hkv, D, dtype, fill_bits=cache.fill_bits)
    saved_gpu, saved_cpu = {}, {}
    scaler, parked_cpu = None, []
    shaped = []
    worst = 0.0
    stale = False
    sc = None if scale == 0.0 else scale
    for op in ops:
        kind = op[0]
        if kind == "embed":
            _, slots, lens, qids = op
            srcs = [dev.prefill(q, n) for q, n in zip(qids, lens)]
            cache.embed(slots, lens, [x[0] for x in srcs], [x[1] for x in srcs])
            hs = [(gen.prefill_host(w.seed, "k", q, NL, Hkv, n, D, dtype),
                   gen.prefill_host(w.seed, "v", q, NL, Hkv, n, D, dtype)) for q, n in zip(qids, lens)]
            pb.embed(slots, lens, [h[0] for h in hs], [h[1] for h in hs])
        elif kind == "evict":
            release, scrub = (op[2], op[3]) if len(op) > 2 else (True, True)
            cache.evict(op[1], release=release, scrub=scrub)
            pb.evict(op[1], release=release)
            stale |= bool(op[1]) and not scrub
        elif kind == "extract":
            _, slots, tag = op
            ks, vs = cache.extract(slots)
            want = pb.extract(slots)
            for (kw, vw), kg, vg in zip(want, ks, vs):
                assert np.array_equal(host_bits(kg), kw) and np.array_equal(host_bits(vg), vw), \
                    f"extract {slots}: bits differ"
            saved_gpu[tag], saved_cpu[tag] = (ks, vs), want
        elif kind == "embed_saved":
            _, slots, tag = op
            ks, vs = saved_gpu[tag]
            cache.embed(slots, [k.shape[2] for k in ks], ks, vs)
            pb.embed(slots, [k.shape[2] for k, _ in saved_cpu[tag]], [k for k, _ in saved_cpu[tag]],
                     [v for _, v in saved_cpu[tag]])
        elif kind == "move":
            cache.move(op[1], op[2])
            pb.move(op[1], op[2])
        elif kind == "shape":
            _, slots, lens, qids = op
            cache.shape_insert(slots, lens)
            pb.shape_insert(slots, lens)
            shaped = list(zip(slots, qids, lens))
        elif kind == "step":
            s = op[1]
            m = cache.build_mask()
            assert np.array_equal(m.cpu().numpy(), pb.mask()), f"{op}: mask"
            for layer in range(NL):
                if shaped:
                    T = pb.step_width()
                    q, kn, vn = dev.prefill_step(s, layer, T, shaped)
                    out = torch.full_like(q, float("nan"))   # positions without a token stay NaN
                    cache.decode_attn(layer, q, kn, vn, out=out, scale=scale)
                    hq = [gen.prefill_step_host(w.seed, which, s, layer, NL, B, T, h, D, dtype, shaped)
                          for which, h in (("q", Hq), ("k", Hkv), ("v", Hkv))]
                    assert np.array_equal(host_bits(kn), hq[1]), "device and host generators disagree"
                    want = pb.decode_layer(layer, *hq, scale=sc)
                    got = O.widen(host_bits(out), dtype)
                    hole = np.isnan(want)
                    assert np.all(np.isnan(got[hole])), f"{op} layer {layer}: a position without a token was written"
                    err = float(np.max(np.abs(got[~hole] - want[~hole]))) if (~hole).any() else 0.0
                else:
                    q, kn, vn = dev.decode(s, layer)
                    out = cache.decode_attn(layer, q, kn, vn, scale=scale)
                    hq = [gen.decode_host(w.seed, sid, s, layer, NL, B, h, D, dtype)
                          for sid, h in ((gen.S_Q, Hq), (gen.S_KNEW, Hkv), (gen.S_VNEW, Hkv))]
                    want = pb.decode_layer(layer, *hq, scale=sc)
                    err = max_err(out, want, dtype)
                worst = max(worst, err)
                assert err <= TOL[dtype], f"{op} layer {layer}: {err}"
            cache.advance()
            pb.advance()
            shaped = []
        elif kind == "flush":
            cache.flush()
        elif kind == "scale":
            from paper_2410_18701_amd.scaling import BatchScaler
            if scaler is None:
                scaler = BatchScaler(cache, op[1])
            scaler.max_cells = op[1]
            parked = scaler.shrink()
            for b in parked:                     # the oracle, in the same order
                parked_cpu.append(pb.extract([b])[0])
                pb.evict([b], release=True)
            if len(op) > 2 and op[2]:
                scaler.prefetch()
            back = scaler.grow()
            for b in back:
                kh, vh = parked_cpu.pop(0)
                pb.embed([b], [kh.shape[2]], [kh], [vh])
            if log is not None:
                log.append(("scale", parked, back))
        else:
            raise ValueError(kind)
        torch.cuda.synchronize()
        check_ring(cache, pb, str(op),
                   live_only=kind in ("evict", "embed", "embed_saved", "extract", "shape", "move", "scale"),
                   tokens_only=stale)
        want_tok = [pb.hist_k[b].shape[2] if pb.lens[b] > 0 else 0 for b in range(B)]
        assert cache.tokens() == want_tok, (op, cache.tokens(), want_tok)
    cache.close()
    note_margin(worst, dtype, f"script {dtype} {NL}x{B}x{Hq}/{Hkv}x{D}")
    return worst
