"""baton_decode_attn_noalloc (GPU): the decode attention without a workspace
argument, its work list and partial sums in the library's static scratch.
Called through the C ABI on one batch and then on a smaller one, its outputs
and caches equal those of baton_decode_attn with a caller workspace bit for
bit, and the oracle's within tolerance; a step too large for the scratch is
refused before anything is enqueued."""
import numpy as np
import pytest
import torch

import oracle.baton_oracle as O
from paper_2410_18701_amd import baton as B
from tests import parity
from workload import configs, driver, gen

pytestmark = pytest.mark.gpu


def _twin_steps(w, split=None, steps=None):
    """The schedule on two identical caches, one decoding through the
    workspace entry point, the other through the no-allocation one."""
    a, dev = driver.open_cache(w, split=split)
    b, _ = driver.open_cache(w, split=split)
    for s, ev in enumerate(w.steps if steps is None else w.steps[:steps]):
        for c in (a, b):
            c.evict(ev.evict, release=True)
        srcs = [dev.prefill(q, n) for q, n in zip(ev.insert_qids, ev.insert_lens)]
        for c in (a, b):
            c.embed(ev.insert, ev.insert_lens, [x[0] for x in srcs], [x[1] for x in srcs])
        L, _, lens = a.query()
        for layer in range(w.n_layers):
            q, kn, vn = dev.decode(s, layer)
            want = a.decode_attn(layer, q, kn, vn)
            got = torch.full_like(q, float("nan"))
            B.baton_decode_attn_noalloc(b.handle, layer, q, kn, vn, got, 0.0,
                                        torch.cuda.current_stream().cuda_stream)
            gb, wb = parity.host_bits(got), parity.host_bits(want)
            assert np.array_equal(gb, wb), f"step {s} layer {layer}: outputs differ"
        for c in (a, b):
            c.advance()
    torch.cuda.synchronize()
    for x, y in ((a.k, b.k), (a.v, b.v)):
        assert torch.equal(x.view(torch.int16), y.view(torch.int16)), "caches differ"
    a.close()
    b.close()


def test_noalloc_matches_workspace_entry_point_then_smaller():
    # a larger batch first: GQA 8:1, 64-token splits (many items per row, the combine)
    big = configs.small("bf16", 2, 16, 16, 2, 128, L0=1500, n_steps=3, n_evict=4, seed=61)
    print("[noalloc] big: bf16 2 layers, 16 slots, GQA 16/2, L0 1500, split 64", flush=True)
    _twin_steps(big, split=64)
    # then a smaller input on the same scratch: MHA, fewer and shorter rows
    small = configs.small("bf16", 1, 4, 4, 4, 64, L0=200, n_steps=2, n_evict=1, seed=62)
    print("[noalloc] small: bf16 1 layer, 4 slots, MHA 4, L0 200", flush=True)
    _twin_steps(small)


def test_noalloc_against_oracle():
    """Whole schedule through the no-allocation entry point, against the
    materialized oracle (fp32, tolerance 1e-5)."""
    w = configs.small("f32", 2, 5, 8, 2, 128, L0=300, n_steps=3, n_evict=2, seed=63)
    print("[noalloc] oracle lockstep: f32 2 layers, 5 slots, GQA 8/2, L0 300", flush=True)
    cache, dev = driver.open_cache(w, split=64)
    pb = O.PaddedBatch(w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.dtype,
                       fill_bits=cache.fill_bits)
    hs = [(gen.prefill_host(w.seed, "k", q, w.n_layers, w.n_kv_heads, w.init_lens[q], w.head_dim, w.dtype),
           gen.prefill_host(w.seed, "v", q, w.n_layers, w.n_kv_heads, w.init_lens[q], w.head_dim, w.dtype))
          for q in range(w.batch)]
    pb.embed(list(range(w.batch)), w.init_lens, [h[0] for h in hs], [h[1] for h in hs])
    worst = 0.0
    for s, ev in enumerate(w.steps):
        cache.evict(ev.evict, release=True)
        pb.evict(ev.evict, release=True)
        srcs = [dev.prefill(q, n) for q, n in zip(ev.insert_qids, ev.insert_lens)]
        cache.embed(ev.insert, ev.insert_lens, [x[0] for x in srcs], [x[1] for x in srcs])
        hs = [(gen.prefill_host(w.seed, "k", q, w.n_layers, w.n_kv_heads, n, w.head_dim, w.dtype),
               gen.prefill_host(w.seed, "v", q, w.n_layers, w.n_kv_heads, n, w.head_dim, w.dtype))
              for q, n in zip(ev.insert_qids, ev.insert_lens)]
        pb.embed(ev.insert, ev.insert_lens, [h[0] for h in hs], [h[1] for h in hs])
        for layer in range(w.n_layers):
            q, kn, vn = dev.decode(s, layer)
            out = torch.empty_like(q)
            B.baton_decode_attn_noalloc(cache.handle, layer, q, kn, vn, out, 0.0,
                                        torch.cuda.current_stream().cuda_stream)
            hq = [gen.decode_host(w.seed, sid, s, layer, w.n_layers, w.batch, h, w.head_dim, w.dtype)
                  for sid, h in ((gen.S_Q, w.n_q_heads), (gen.S_KNEW, w.n_kv_heads), (gen.S_VNEW, w.n_kv_heads))]
            want = pb.decode_layer(layer, hq[0], hq[1], hq[2])
            err = parity.max_err(out, want, w.dtype)
            worst = max(worst, err)
            assert err <= parity.TOL[w.dtype], f"step {s} layer {layer}: {err}"
        cache.advance()
        pb.advance()
        torch.cuda.synchronize()
        parity.check_ring(cache, pb, f"step {s}")
    cache.close()
    parity.note_margin(worst, w.dtype, "no-allocation entry point")


def test_noalloc_holey_rows():
    """In-batch prefill steps (no prefill/decode separation) through the
    no-allocation entry point: holey rows whose one-token runs are read as
    gathered items (MHA bf16, the VALU kernel), and the prompts' prefill --
    bit for bit the workspace entry point's outputs and caches."""
    w = configs.small("bf16", 1, 6, 8, 8, 128, L0=150, n_steps=14, n_evict=1, new_hi=60, seed=64)
    print("[noalloc] holey rows: bf16 1 layer, 6 slots, MHA 8, L0 150, a prefill every step", flush=True)
    a, dev = driver.open_cache(w, no_pd=True)
    b, _ = driver.open_cache(w, no_pd=True)
    st = torch.cuda.current_stream().cuda_stream
    for s, ev in enumerate(w.steps):
        ins = list(zip(ev.insert, ev.insert_qids, ev.insert_lens))
        for c in (a, b):
            c.evict(ev.evict, release=True)
            if ins:
                c.shape_insert(ev.insert, ev.insert_lens)
        T = a.step_width
        for layer in range(w.n_layers):
            q, kn, vn = dev.prefill_step(s, layer, T, ins) if ins else dev.decode(s, layer)
            want = torch.zeros_like(q)
            a.decode_attn(layer, q, kn, vn, out=want)
            got = torch.zeros_like(q)
            B.baton_decode_attn_noalloc(b.handle, layer, q, kn, vn, got, 0.0, st)
            assert np.array_equal(parity.host_bits(got), parity.host_bits(want)), f"step {s} layer {layer}"
        for c in (a, b):
            c.advance()
    torch.cuda.synchronize()
    for x, y in ((a.k, b.k), (a.v, b.v)):
        assert torch.equal(x.view(torch.int16), y.view(torch.int16)), "caches differ"
    a.close()
    b.close()


def test_noalloc_refuses_a_step_beyond_the_scratch():
    """512 slots of 3000 tokens, 8 kv-heads of 8 q-heads, 64-token splits:
    about 24,000 items per kv-head, far beyond the scratch.  ESCRATCH, nothing
    enqueued, the layer still to be decoded; the workspace entry point (and
    the no-allocation one after a larger split) then decode it."""
    NL, Bt, Hq, Hkv, D, n = 1, 512, 64, 8, 128, 3000
    cache = driver.BatonCache(NL, Bt, Hq, Hkv, D, n + 64, dtype="bf16")
    src = torch.randn((NL, Hkv, n, D), device="cuda").to(torch.bfloat16)
    cache.embed(list(range(Bt)), [n] * Bt, [src] * Bt, [src] * Bt)
    cache.set_split_tokens(64)
    q = torch.randn((Bt, Hq, D), device="cuda").to(torch.bfloat16)
    kn = torch.randn((Bt, Hkv, D), device="cuda").to(torch.bfloat16)
    out = torch.full_like(q, float("nan"))
    st = torch.cuda.current_stream().cuda_stream
    with pytest.raises(B.BatonError) as e:
        B.baton_decode_attn_noalloc(cache.handle, 0, q, kn, kn, out, 0.0, st)
    assert e.value.status == B.BATON_ESCRATCH
    torch.cuda.synchronize()
    assert torch.isnan(out.float()).all(), "nothing may have been written"
    cache.flush()
    with pytest.raises(B.BatonError):
        cache.advance()                               # the layer is still to be decoded
    want = cache.decode_attn(0, q, kn, kn)
    cache.advance()
    cache.set_split_tokens(4096)
    got = torch.empty_like(q)
    B.baton_decode_attn_noalloc(cache.handle, 0, q, kn, kn, got, 0.0, st)
    torch.cuda.synchronize()
    assert torch.isfinite(got.float()).all() and torch.isfinite(want.float()).all()
    cache.close()
