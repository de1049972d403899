"""Feeds a Workload through libbaton on the GPU (test and benchmark harness).

Inputs are generated in device memory by the workload generator (the same
values the host generator gives the oracle).  The step sequence is the one
the paper's P&D insertion implies: evict finished queries (releasing shared
leading placeholders), embed the newly prefilled ones, build the mask, run
decode attention layer by layer, advance.
"""
import torch

from paper_2410_18701_amd.cache import BatonCache, torch_dtype

from . import gen


class DeviceInputs:
    """Device tensors of one workload's generated inputs."""

    def __init__(self, w, device="cuda"):
        self.w = w
        self.device = device
        self.tdt = torch_dtype(w.dtype)

    def _fill(self, t, stream_id, shape, c0, strides):
        gen.fill_device(t.data_ptr(), self.w.seed, stream_id, self.w.dtype, shape, c0, strides,
                        torch.cuda.current_stream().cuda_stream)

    def prefill(self, qid, length):
        """(k, v) of a prefilled query: [n_layers][n_kv_heads][length][head_dim]."""
        w = self.w
        shape = (w.n_layers, w.n_kv_heads, length, w.head_dim)
        out = []
        for sid in (gen.S_PREFILL_K, gen.S_PREFILL_V):
            t = torch.empty(shape, dtype=self.tdt, device=self.device)
            c0, st = gen.prefill_counter(qid, w.n_layers, w.n_kv_heads, w.head_dim)
            self._fill(t, sid, shape, c0, st)
            out.append(t)
        return out

    def decode(self, step, layer):
        """(q, k_new, v_new) of one layer of one step."""
        w = self.w
        out = []
        for sid, heads in ((gen.S_Q, w.n_q_heads), (gen.S_KNEW, w.n_kv_heads), (gen.S_VNEW, w.n_kv_heads)):
            t = torch.empty((w.batch, heads, w.head_dim), dtype=self.tdt, device=self.device)
            c0, st = gen.decode_counter(step, layer, w.n_layers, w.batch, heads, w.head_dim)
            self._fill(t, sid, (1, w.batch, heads, w.head_dim), c0, st)
            out.append(t)
        return out


    def prefill_step(self, step, layer, T, inserted=()):
        """(q, k_new, v_new) of one layer of a step that prefills queries inside
        the batch: [batch][T][heads][head_dim]; inserted as in gen.prefill_step_host."""
        w = self.w
        out = []
        for sid, psid, heads in ((gen.S_QW, None, w.n_q_heads), (gen.S_KW, gen.S_PREFILL_K, w.n_kv_heads),
                                 (gen.S_VW, gen.S_PREFILL_V, w.n_kv_heads)):
            t = torch.empty((w.batch, T, heads, w.head_dim), dtype=self.tdt, device=self.device)
            c0, st = gen.wide_counter(step, layer, w.n_layers, w.batch, heads, w.head_dim)
            self._fill(t, sid, (w.batch, T, heads, w.head_dim), c0, st)
            if psid is not None:
                for slot, qid, n in inserted:
                    c0, st = gen.prompt_counter(qid, layer, w.n_layers, heads, w.head_dim)
                    self._fill(t[slot, T - n:], psid, (1, n, heads, w.head_dim), c0, st)
            out.append(t)
        return out


def prefill_bytes(w, length):
    return 2 * w.n_layers * w.n_kv_heads * length * w.head_dim * w.elem_bytes


def open_cache(w, capacity=None, device="cuda", fill_bits=None, split=None, init_budget=8 << 30,
               no_pd=False):
    """A BatonCache holding the workload's initial batch, built by embedding the
    B initial queries (query id = slot) into an empty batch, a group at a time."""
    if capacity is None:
        capacity = w.capacity_no_pd() if no_pd else w.capacity()
    cap = capacity
    cache = BatonCache(w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, cap,
                       dtype=w.dtype, fill_bits=fill_bits, device=device)
    if split is not None:
        cache.set_split_tokens(split)
    inputs = DeviceInputs(w, device)
    group, used = [], 0
    for b in range(w.batch):
        group.append(b)
        used += prefill_bytes(w, w.init_lens[b])
        if used >= init_budget or b == w.batch - 1:
            srcs = [inputs.prefill(q, w.init_lens[q]) for q in group]
            cache.embed(group, [w.init_lens[q] for q in group], [s[0] for s in srcs], [s[1] for s in srcs])
            torch.cuda.current_stream().synchronize()
            del srcs
            group, used = [], 0
    return cache, inputs


def run_step_no_pd(cache, inputs, s, ev, mask=True):
    """Step s without prefill/decode separation: evict, register the new queries
    for prefill inside the batch, mask, every layer (prefill-step inputs when
    there are new queries), advance."""
    w = inputs.w
    cache.evict(ev.evict, release=True)
    inserted = list(zip(ev.insert, ev.insert_qids, ev.insert_lens))
    if inserted:
        cache.shape_insert(ev.insert, ev.insert_lens)
    T = cache.step_width
    m = cache.build_mask() if mask else None
    for layer in range(w.n_layers):
        q, kn, vn = inputs.prefill_step(s, layer, T, inserted) if inserted else inputs.decode(s, layer)
        cache.decode_attn(layer, q, kn, vn)
    cache.advance()
    return m


def run_step(cache, inputs, s, ev, layers=None, outs=None, mask=True):
    """Step s of the schedule: evict, embed, mask, decode every layer, advance.

    Returns (mask tensor or None, list of per-layer outputs if outs is a list).
    """
    w = inputs.w
    cache.evict(ev.evict, release=True)
    if ev.insert:
        srcs = [inputs.prefill(q, n) for q, n in zip(ev.insert_qids, ev.insert_lens)]
        cache.embed(ev.insert, ev.insert_lens, [x[0] for x in srcs], [x[1] for x in srcs])
    m = cache.build_mask() if mask else None
    for layer in range(w.n_layers) if layers is None else layers:
        q, kn, vn = inputs.decode(s, layer)
        o = cache.decode_attn(layer, q, kn, vn)
        if outs is not None:
            outs.append((layer, q, kn, vn, o))
    cache.advance()
    return m
