"""The synthetic decode workloads and their seeded event schedules.

A workload is a batch of B slots decoding together.  Its schedule says, for
each decode step, which slots' queries finish (emit EOS) and which new,
already-prefilled queries take the freed slots, with their prefilled lengths.
Lengths and events are host integers drawn from the S_LENS / S_EVENTS streams
of workload/gen.py; tensor values are drawn by the tensor generator from the
query id (prefill K/V) or from (step, layer, slot, head) (decode inputs).

The paper evaluates on two simulated query sets it did not release (long-in /
short-out, short-in / long-out and short/short queries of a few dozen to about
4,000 words).  These workloads stand in for them: the length laws cover the
same spans, and 7b-b64-L4096 has the attention shape of the 7B model it serves
(32 layers x 32 heads x 128).
"""
import math
from dataclasses import dataclass, field
from typing import List, Optional

from . import gen


class Draws:
    """Sequential consumer of one generator stream (host integers and floats)."""

    def __init__(self, seed, stream):
        self.key = gen.stream_key(seed, stream)
        self.j = 0

    def u64(self):
        v = gen.draw(self.key, self.j)
        self.j += 1
        return v

    def uniform01(self):
        """Uniform on [0, 1) with 53 random bits."""
        return (self.u64() >> 11) * 2.0 ** -53

    def randint(self, lo, hi):
        """Uniform integer on [lo, hi]."""
        return lo + (((self.u64() >> 11) * (hi - lo + 1)) >> 53)

    def normal(self):
        """Standard normal by Box-Muller (host-only: lengths, never tensor values)."""
        u1 = ((self.u64() >> 11) + 1) * 2.0 ** -53
        u2 = self.uniform01()
        return math.sqrt(-2.0 * math.log(u1)) * math.cos(2.0 * math.pi * u2)

    def lognormal_int(self, mu, sigma, lo, hi):
        return int(min(hi, max(lo, round(math.exp(mu + sigma * self.normal())))))

    def poisson(self, lam):
        """Knuth's product-of-uniforms method."""
        limit, k, p = math.exp(-lam), 0, 1.0
        while True:
            p *= self.uniform01()
            if p <= limit:
                return k
            k += 1

    def sample(self, items, k):
        """k distinct items, uniformly (partial Fisher-Yates), returned sorted."""
        pool = list(items)
        for i in range(k):
            j = i + self.randint(0, len(pool) - 1 - i)
            pool[i], pool[j] = pool[j], pool[i]
        return sorted(pool[:k])


@dataclass
class StepEvents:
    evict: List[int]          # slots whose queries finished, ascending
    insert: List[int]         # slots that take new queries, ascending
    insert_lens: List[int]    # prefilled length of each new query
    insert_qids: List[int]    # query id of each new query


@dataclass
class Workload:
    name: str
    dtype: str                # "f32" or "bf16"
    n_layers: int
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    L0: int                   # padded length of the initial batch
    n_steps: int
    seed: int
    init_lens: List[int] = field(default_factory=list)   # qid of slot b is b
    steps: List[StepEvents] = field(default_factory=list)
    note: str = ""

    @property
    def elem_bytes(self):
        return 4 if self.dtype == "f32" else 2

    def capacity(self, extra_steps=0):
        """Ring columns per row: room for the longest padded length the run can reach.

        Every prefilled length here is at most L0, so the padded length can
        only pass L0 through one appended column per step.
        """
        need = max(self.L0, max(self.init_lens, default=0),
                   max((max(e.insert_lens, default=0) for e in self.steps), default=0))
        cap = need + self.n_steps + extra_steps + 1
        return (cap + 63) // 64 * 64

    def capacity_no_pd(self):
        """Ring columns when the new queries are prefilled inside the batch: a step
        with insertions appends as many columns as its longest prompt."""
        need = max(self.L0, max(self.init_lens, default=0))
        cap = need + sum(max(e.insert_lens, default=1) for e in self.steps) + 1
        return (cap + 63) // 64 * 64


def _pin_max(lens, L0):
    """Give the longest drawn row exactly L0 columns (the batch's padded length)."""
    i = max(range(len(lens)), key=lambda b: lens[b])
    lens[i] = L0
    return lens


def _schedule(w: Workload, n_evict, new_len, d: Draws):
    live = set(range(w.batch))
    next_qid = w.batch
    for _ in range(w.n_steps):
        k = min(n_evict(d), len(live))
        ev = d.sample(sorted(live), k)
        lens = [new_len(d) for _ in ev]
        qids = list(range(next_qid, next_qid + k))
        next_qid += k
        w.steps.append(StepEvents(evict=ev, insert=list(ev), insert_lens=lens, insert_qids=qids))
    return w


def tiny_f32():
    """fp32, 1 layer, B=4, 4 heads, D=64, L=128; one EOS in slot 2 replaced by a 40-token query."""
    w = Workload("tiny-f32", "f32", 1, 4, 4, 4, 64, 128, 1, seed=1001)
    d = Draws(w.seed, gen.S_LENS)
    w.init_lens = _pin_max([d.randint(16, 128) for _ in range(w.batch)], w.L0)
    w.steps = [StepEvents(evict=[2], insert=[2], insert_lens=[40], insert_qids=[w.batch])]
    return w


def b32_l2048(n_steps=16):
    """bf16, 1 layer, B=32, 32 heads, D=128, L=2048; 2 EOS + 2 inserts of U[64,1024] per step."""
    w = Workload("b32-L2048", "bf16", 1, 32, 32, 32, 128, 2048, n_steps, seed=1002)
    d = Draws(w.seed, gen.S_LENS)
    w.init_lens = _pin_max([d.randint(128, 2048) for _ in range(w.batch)], w.L0)
    return _schedule(w, lambda _d: 2, lambda e: e.randint(64, 1024), Draws(w.seed, gen.S_EVENTS))


def llama7b_b64_l4096(n_steps=64):
    """bf16, 32 layers x 32 heads x 128 (7B-shaped), B=64, L=4096; lognormal lengths, Poisson(4) arrivals."""
    w = Workload("7b-b64-L4096", "bf16", 32, 64, 32, 32, 128, 4096, n_steps, seed=1003)
    d = Draws(w.seed, gen.S_LENS)
    w.init_lens = _pin_max([d.lognormal_int(6.5, 0.8, 32, 4096) for _ in range(w.batch)], w.L0)
    return _schedule(w, lambda e: e.poisson(4.0), lambda e: e.lognormal_int(6.5, 0.8, 32, 4096),
                     Draws(w.seed, gen.S_EVENTS))


def gqa70b_b128_l8192(n_steps=16, n_layers=80):
    """bf16, GQA 64 q-heads / 8 KV heads, D=128, 80 layers, B=128, L=8192; 8 EOS + 8 inserts per step."""
    w = Workload("70b-gqa-b128-L8192", "bf16", n_layers, 128, 64, 8, 128, 8192, n_steps, seed=1004)
    d = Draws(w.seed, gen.S_LENS)
    w.init_lens = _pin_max([d.randint(256, 8192) for _ in range(w.batch)], w.L0)
    return _schedule(w, lambda _d: 8, lambda e: e.randint(256, 8192), Draws(w.seed, gen.S_EVENTS))


def skew_b256_l32768(n_steps=16):
    """Long-skew: bf16, 1 layer, B=256, 32 heads, D=128, L=32768; 90% U[64,1024], 10% U[16384,32768]."""
    w = Workload("skew-b256-L32768", "bf16", 1, 256, 32, 32, 128, 32768, n_steps, seed=1005)
    d = Draws(w.seed, gen.S_LENS)
    n_long = round(0.1 * w.batch)
    long_rows = set(d.sample(range(w.batch), n_long))
    lens = [d.randint(16384, 32768) if b in long_rows else d.randint(64, 1024)
            for b in range(w.batch)]
    w.init_lens = _pin_max(lens, w.L0)
    return _schedule(w, lambda _d: 4, lambda e: e.randint(64, 16384), Draws(w.seed, gen.S_EVENTS))


def skew_growth_b256_l32768(n_steps=16):
    """Long-skew growth variant: the long rows finish at step 0, then each step inserts a query
    longer than the padded length (1024 + s*960 tokens), so every insert grows the batch."""
    w = skew_b256_l32768(0)
    w.name, w.n_steps = "skew-growth-b256-L32768", n_steps + 1
    d = Draws(w.seed, gen.S_EVENTS)
    long_rows = [b for b in range(w.batch) if w.init_lens[b] > 1024]
    next_qid = w.batch
    lens0 = [d.randint(64, 1024) for _ in long_rows]
    w.steps.append(StepEvents(long_rows, list(long_rows), lens0,
                              list(range(next_qid, next_qid + len(long_rows)))))
    next_qid += len(long_rows)
    live = set(range(w.batch))
    for s in range(1, n_steps + 1):
        ev = d.sample(sorted(live), 1)
        w.steps.append(StepEvents(ev, list(ev), [1024 + s * 960], [next_qid]))
        next_qid += 1
    return w


def small(dtype="bf16", n_layers=2, batch=5, n_q_heads=4, n_kv_heads=2, head_dim=64, L0=300,
          n_steps=4, n_evict=2, len_lo=1, len_hi=None, seed=7, new_hi: Optional[int] = None):
    """A small random workload for parity tests: sizes the oracle finishes in seconds."""
    w = Workload(f"small-{dtype}-{n_layers}x{batch}x{n_q_heads}/{n_kv_heads}x{head_dim}-L{L0}",
                 dtype, n_layers, batch, n_q_heads, n_kv_heads, head_dim, L0, n_steps, seed=seed)
    d = Draws(seed, gen.S_LENS)
    hi = L0 if len_hi is None else len_hi
    w.init_lens = _pin_max([d.randint(len_lo, hi) for _ in range(batch)], L0)
    nh = L0 if new_hi is None else new_hi
    return _schedule(w, lambda _d: n_evict, lambda e: e.randint(1, nh), Draws(seed, gen.S_EVENTS))


# The workloads by name (the name each builds its Workload with).
CONFIGS = {"tiny-f32": tiny_f32, "b32-L2048": b32_l2048, "7b-b64-L4096": llama7b_b64_l4096,
           "70b-gqa-b128-L8192": gqa70b_b128_l8192, "skew-b256-L32768": skew_b256_l32768,
           "skew-growth-b256-L32768": skew_growth_b256_l32768}
