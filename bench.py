"""Benchmark of the re-batched decode step on one MI355X.

One step = the whole hot path over the batch: evict the queries that finished
(placeholders over their tokens, release of shared leading placeholders),
embed the newly prefilled queries end-aligned (growing the batch on the left
when one is longer), build the mask, then masked decode attention layer by
layer (appending each layer's new key/value column), then advance.

Default workload (70b-gqa-b128-L8192), the largest configuration: bf16,
grouped-query attention with 64 query heads over 8 kv-heads, head_dim 128,
batch 128, initial padded length 8192, lengths uniform in [256, 8192], 8
queries finishing and 8 prefilled queries inserted per step.  The dense
padded cache of all 80 layers (343.6 GB) exceeds the GPU's 288 GB, so 24 of
the 80 layers are resident and each step decodes those 24, each at the real
per-layer shape.  All inputs are synthetic and seeded, generated into HBM
before the timed region.  The 7B-shaped workload (7b-b64-L4096: 32 layers x 32
heads, batch 64, L 4096) runs after it and is reported under "also".

Prints one JSON line: query-tokens/s of whole steps, the dominant kernel's
roofline (decode attention, HBM-bound), per-op HBM GB/s (kv_embed with and
without the placeholder writes of scrubbing evictions), and the CPU oracle
timed on a bounded sample on this host's cores.
"""
import argparse
import gc
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
GQA_WORKLOAD = "70b-gqa-b128-L8192"   # 80 layers' padded cache exceed HBM: a resident subset
GQA_LAYERS, GQA_RESIDENT = 80, 24
DEFAULT_WORKLOAD = GQA_WORKLOAD
SECONDARY_WORKLOAD = "7b-b64-L4096"
NO_PD_WORKLOAD = "b32-L2048"   # without P&D separation every step widens the ring by its longest prompt
# rocprofv3 FETCH_SIZE / WRITE_SIZE records of decode attention, by workload:
# traffic over algorithmic bytes, valid for the kernel sources they were taken on
TRAFFIC = {GQA_WORKLOAD: "decode_attn_70b_gqa_b128_L8192_traffic.json"}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=4)
    p.add_argument("--config", default=None,
                   choices=["b32-L2048", "7b-b64-L4096", "70b-gqa-b128-L8192", "skew-b256-L32768",
                            "skew-growth-b256-L32768"])
    p.add_argument("--layers", type=int, default=None,
                   help=f"resident layers (70b-gqa-b128-L8192's 80-layer padded cache exceeds HBM; "
                        f"default {GQA_RESIDENT} there)")
    p.add_argument("--split", type=int, default=None, help="tokens per attention work item")
    p.add_argument("--no-pd", action="store_true",
                   help="prefill the new queries inside the batch (no prefill/decode separation) "
                        f"instead of embedding prefilled ones (default workload then {NO_PD_WORKLOAD})")
    p.add_argument("--model", default=None, choices=["llama2-7b"],
                   help="run whole decode layers of this model (synthetic weights) around the attention "
                        f"(default workload then {SECONDARY_WORKLOAD})")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-workers", type=int, default=16,
                   help="most worker processes of the CPU oracle's all-cores run (the host's cores, at most this)")
    p.add_argument("--no-scrub-steps", type=int, default=8,
                   help="steps after the timed ones whose evictions do not scrub, timed for kv_embed alone (0: skip)")
    p.add_argument("--no-secondary", action="store_true",
                   help=f"skip the {SECONDARY_WORKLOAD} run reported under 'also'")
    p.add_argument("--lead-bytes", type=int, default=2 << 30,
                   help="size of the device copy queued ahead of each timed region so that the host loop "
                        "runs ahead of the GPU (0: none)")
    p.add_argument("--copy-bytes", type=int, default=2 << 30,
                   help="size of the plain device copy timed as the achievable-bandwidth reference (0: skip)")
    p.add_argument("--traffic-dir", default=os.path.join(ROOT, "profiles"),
                   help="where the rocprofv3-derived traffic records of decode attention are (FETCH_SIZE/"
                        "WRITE_SIZE scaled by a copy of known size, as a ratio to the algorithmic bytes); a "
                        "record is used only for its workload and while the kernel sources are unchanged")
    args = p.parse_args()
    if args.config is None:
        args.config = SECONDARY_WORKLOAD if args.model else NO_PD_WORKLOAD if args.no_pd else DEFAULT_WORKLOAD
    return args


def log(msg):
    """A progress line on stderr (the JSON result is the only line on stdout)."""
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def queue_lead(nbytes):
    """A plain device copy of nbytes queued right before a timed region, outside
    it (the region's first event follows it on the stream): while the GPU
    copies, the host loop (Python, an event pair per operation) enqueues the
    first steps and then stays ahead, so that a one-layer step's short kernels
    do not wait for the host's next launch.  Returns the buffers, to be kept
    until the region has ended."""
    import torch
    if nbytes <= 0:
        return None
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    return src, dst


def attn_bytes(w, lens):
    """Algorithmic HBM bytes of one decode_attn launch: cached K and V of live
    rows, k_new/v_new read and appended, q of live rows, out of every row."""
    sz, D = w.elem_bytes, w.head_dim
    live = [n for n in lens if n > 0]
    kv = 2 * w.n_kv_heads * D * sum(live)
    new = 2 * 2 * w.n_kv_heads * D * len(live)
    qo = w.n_q_heads * D * (len(live) + w.batch)
    return sz * (kv + new + qo)


def embed_bytes(w, insert_lens):
    """Read of the prefilled K/V plus its write into the cache, all layers."""
    return 2 * sum(2 * w.n_layers * w.n_kv_heads * n * w.head_dim * w.elem_bytes for n in insert_lens)


def placeholder_bytes(w, lens_before, ev):
    """Placeholder writes a step owes for its evictions (overhead, not algorithmic):
    an evicted slot that takes a new query owes only the columns in front of it."""
    new = dict(zip(ev.insert, ev.insert_lens))
    owed = sum(max(0, lens_before[s] - new.get(s, 0)) for s in ev.evict)
    return 2 * w.n_layers * w.n_kv_heads * owed * w.head_dim * w.elem_bytes


def prefill_flops(w, insert_lens):
    """Algorithmic flops of the causal prefill attention of new queries, one layer:
    per query head, 2*D flops per (position, visible key) pair for QK^T and the
    same for PV."""
    return sum(4 * w.n_q_heads * w.head_dim * n * (n + 1) // 2 for n in insert_lens)


def bench_no_pd(args, w):
    """The schedule without prefill/decode separation: a step with new queries
    prefills them inside the batch (their prompts as T = longest-prompt input
    positions, the other rows padded), leaving holes in the other rows."""
    import torch

    from workload import driver

    cache, inputs = driver.open_cache(w, split=args.split, no_pd=True)
    total_steps = args.warmup + args.steps
    for s in range(args.warmup):
        driver.run_step_no_pd(cache, inputs, s, w.steps[s])
    torch.cuda.synchronize()
    pre = []
    for s in range(args.warmup, total_steps):
        ev = w.steps[s]
        ins = list(zip(ev.insert, ev.insert_qids, ev.insert_lens))
        T = max(ev.insert_lens, default=1)
        dec = [inputs.prefill_step(s, layer, T, ins) if ins else inputs.decode(s, layer)
               for layer in range(w.n_layers)]
        outs = torch.empty_like(dec[0][0])
        pre.append((ins, dec, outs))
    mask_buf = torch.empty((w.batch, cache.capacity + 1), dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    n_ev = 2 * args.steps * (2 + w.n_layers) + 2
    pool = [torch.cuda.Event(enable_timing=True) for _ in range(n_ev)]
    for e in pool:
        e.record()
    torch.cuda.synchronize()
    pool_it = iter(pool)
    E = lambda: next(pool_it)
    ev_pf, ev_dec = [], []
    bytes_dec = flops_pf = 0
    live_tokens = prompt_tokens = 0
    gc.collect()
    gc.disable()
    t_start, t_end = E(), E()
    lead = queue_lead(args.lead_bytes)
    t_start.record()
    for i, s in enumerate(range(args.warmup, total_steps)):
        ev = w.steps[s]
        ins, dec, outs = pre[i]
        cache.evict(ev.evict, release=True)
        if ins:
            cache.shape_insert(ev.insert, ev.insert_lens)
        cache.build_mask(out=mask_buf)
        _, _, lens = cache.query()
        for layer in range(w.n_layers):
            q, kn, vn = dec[layer]
            a, b = E(), E()
            a.record()
            cache.decode_attn(layer, q, kn, vn, out=outs)
            b.record()
            (ev_pf if ins else ev_dec).append((a, b))
        if ins:
            flops_pf += w.n_layers * prefill_flops(w, ev.insert_lens)
            prompt_tokens += sum(ev.insert_lens)
        else:
            bytes_dec += w.n_layers * attn_bytes(w, lens)
        live_tokens += sum(1 for n in lens if n > 0) + len(ins)
        cache.advance()
    t_end.record()
    torch.cuda.synchronize()
    del lead
    gc.enable()
    total_ms = t_start.elapsed_time(t_end)
    ms = lambda evs: sum(x.elapsed_time(y) for x, y in evs)
    pf_ms, dec_ms = ms(ev_pf), ms(ev_dec)
    L, _, _ = cache.query()
    return {
        "metric": "query-tokens/s without prefill/decode separation (new queries prefilled in the batch)",
        "value": round(live_tokens / (total_ms * 1e-3), 1),
        "unit": "query-tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(total_ms / args.steps, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic (seeded counter-based generator, values ~N(0,1))",
        "config": {"workload": f"{w.name} schedule, no P&D separation: {w.dtype}, {w.n_layers} layers x "
                               f"{w.n_q_heads} q-heads / {w.n_kv_heads} kv-heads x head_dim {w.head_dim}, "
                               f"batch {w.batch}, initial padded length {w.L0}, ring capacity {cache.capacity}",
                   "global_batch": w.batch, "seq_len": w.L0, "parallelism": "none (1 GPU)"},
        "ops": {
            "prefill_steps": {"layer_calls": len(ev_pf), "ms_per_call": round(pf_ms / max(1, len(ev_pf)), 4),
                              "prompt_tokens": prompt_tokens,
                              "call_ms": quantiles([x.elapsed_time(y) for x, y in ev_pf]),
                              "prefill_TFLOP/s (calls incl. decode rows)":
                                  round(flops_pf / (pf_ms * 1e-3) / 1e12, 2) if pf_ms else None},
            "decode_steps": {"layer_calls": len(ev_dec), "ms_per_call": round(dec_ms / max(1, len(ev_dec)), 4),
                             "call_ms": quantiles([x.elapsed_time(y) for x, y in ev_dec]),
                             "GB/s": round(bytes_dec / (dec_ms * 1e-3) / 1e9, 1) if dec_ms else None},
            "final_padded_length": L,
        },
    }


def bench_model(args, w):
    """Whole decode steps of a llama2-7b-shaped model on the workload's schedule:
    evict, embed, mask, then per layer RMS norm, QKV projection, rotary
    embedding, the re-batched attention, output projection, RMS norm, gated
    feed-forward; synthetic weights resident in HBM."""
    import torch

    from paper_2410_18701_amd import layer as PL
    from workload import driver
    from workload import model as M

    m = M.LLAMA2_7B
    if (w.n_q_heads, w.n_kv_heads, w.head_dim) != (m.n_q_heads, m.n_kv_heads, m.head_dim):
        raise SystemExit("--model llama2-7b needs a workload with 32 heads of 128 (b32-L2048, 7b-b64-L4096, "
                         "skew-b256-L32768)")
    cache, inputs = driver.open_cache(w, split=args.split)
    weights = [M.weights_device(w.seed, m, l) for l in range(w.n_layers)]
    wbytes = sum(t.numel() * 2 for lw in weights for t in lw.values())
    gemm = PL.Gemm()
    layers = PL.DecodeLayers(cache, weights, gemm, m.theta, m.eps)
    total_steps = args.warmup + args.steps
    xs = [M.x_device(w.seed, s, w.batch, m.hidden) for s in range(total_steps)]

    def step(s, pre=None, ev_attn=None, ev_layer=None, E=None):
        ev = w.steps[s]
        cache.evict(ev.evict, release=True)
        if ev.insert:
            srcs = pre if pre is not None else [inputs.prefill(q, n) for q, n in zip(ev.insert_qids, ev.insert_lens)]
            cache.embed(ev.insert, ev.insert_lens, [x[0] for x in srcs], [x[1] for x in srcs])
        cache.build_mask(out=mask_buf)
        n_live = sum(1 for n in cache.query()[2] if n > 0)
        x = xs[s]
        for layer in range(w.n_layers):
            if E is not None:
                a = E()
                a.record()
            layers.layer(layer, x)
            if E is not None:
                b = E()
                b.record()
                ev_layer.append((a, b))
        cache.advance()
        return n_live

    mask_buf = torch.empty((w.batch, cache.capacity + 1), dtype=torch.uint8, device="cuda")
    for s in range(args.warmup):
        step(s)
    torch.cuda.synchronize()
    pre = [[inputs.prefill(q, n) for q, n in zip(w.steps[s].insert_qids, w.steps[s].insert_lens)]
           for s in range(args.warmup, total_steps)]
    pool = [torch.cuda.Event(enable_timing=True) for _ in range(2 * args.steps * w.n_layers + 2)]
    for e in pool:
        e.record()
    torch.cuda.synchronize()
    it = iter(pool)
    E = lambda: next(it)
    ev_layer, live_tokens = [], 0
    gc.collect()
    gc.disable()
    t0, t1 = E(), E()
    lead = queue_lead(args.lead_bytes)
    t0.record()
    for i, s in enumerate(range(args.warmup, total_steps)):
        live_tokens += step(s, pre[i], None, ev_layer, E)
    t1.record()
    torch.cuda.synchronize()
    del lead
    gc.enable()
    total_ms = t0.elapsed_time(t1)
    layer_ms = sum(a.elapsed_time(b) for a, b in ev_layer)
    per_layer_w = wbytes / w.n_layers
    gemm.close()
    return {
        "metric": "decode tokens/s of whole llama2-7b-shaped decode steps (synthetic weights)",
        "value": round(live_tokens / (total_ms * 1e-3), 1), "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(total_ms / args.steps, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded generator weights and activations)",
        "config": {"workload": f"{w.name} schedule with llama2-7b layers: {w.n_layers} layers, hidden "
                               f"{m.hidden}, ffn {m.ffn}, batch {w.batch}, initial padded length {w.L0}",
                   "global_batch": w.batch, "seq_len": w.L0, "parallelism": "none (1 GPU)"},
        "ops": {"layer": {"ms_per_call": round(layer_ms / len(ev_layer), 4),
                          "call_ms": quantiles([a.elapsed_time(b) for a, b in ev_layer]),
                          "weight_bytes_per_layer": int(per_layer_w)},
                "weights_GB": round(wbytes / 1e9, 2)},
    }


def _oracle_share(w, share, n_shares, barrier, out):
    """One worker of the CPU baseline (a forked process, one thread): the
    oracle over the slots b with b % n_shares == share of layer 0 of the
    workload's initial batch, then step 0 (evict, embed, mask, attention,
    advance) timed.  Worker 0 first runs its share alone (on a copy), while
    the others wait: the single-thread figure."""
    import copy

    from threadpoolctl import threadpool_limits

    import oracle.baton_oracle as O
    from workload import gen

    with threadpool_limits(limits=1):
        layer = 0
        mine = [b for b in range(w.batch) if b % n_shares == share]
        ev = w.steps[0]
        pb = O.PaddedBatch(1, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.dtype)

        def layer_src(qid, n):
            c0, st = gen.prefill_counter(qid, w.n_layers, w.n_kv_heads, w.head_dim, layer0=layer)
            shp = (1, w.n_kv_heads, n, w.head_dim)
            return (gen.fill_host(w.seed, gen.S_PREFILL_K, w.dtype, shp, c0, st),
                    gen.fill_host(w.seed, gen.S_PREFILL_V, w.dtype, shp, c0, st))

        order = sorted(mine, key=lambda b: -w.init_lens[b])       # the longest first: one growth
        init = [layer_src(b, w.init_lens[b]) for b in order]
        pb.embed(order, [w.init_lens[b] for b in order], [x[0] for x in init], [x[1] for x in init])
        del init
        ev_slots = [b for b in ev.evict if b in mine]
        ins = [(b, q, n) for b, q, n in zip(ev.insert, ev.insert_qids, ev.insert_lens) if b in mine]
        srcs = [layer_src(q, n) for _, q, n in ins]
        dec = [gen.decode_host(w.seed, sid, 0, layer, w.n_layers, w.batch, h, w.head_dim, w.dtype)
               for sid, h in ((gen.S_Q, w.n_q_heads), (gen.S_KNEW, w.n_kv_heads), (gen.S_VNEW, w.n_kv_heads))]

        def step(batch):
            t0 = time.perf_counter()
            batch.evict(ev_slots, release=True)
            batch.embed([b for b, _, _ in ins], [n for _, _, n in ins], [x[0] for x in srcs], [x[1] for x in srcs])
            batch.mask()
            batch.decode_layer(0, dec[0], dec[1], dec[2])
            batch.advance()
            return t0, time.perf_counter(), len(batch.live())

        barrier.wait()
        if share == 0:
            out.put(("solo",) + step(copy.deepcopy(pb)))
        barrier.wait()
        out.put(("all",) + step(pb))


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(w, max_workers):
    """The oracle as it stands, timed on this host's cores over a bounded
    sample of the workload: step 0 of layer 0 (evict, embed, mask, attention,
    advance over the query histories), its 128 slots dealt over worker
    processes of one thread each, all run together (the all-cores figure); the
    first worker's share also run alone (the single-thread figure, scaled by
    the number of shares).  Scaled to query-tokens/s of the benchmark's step
    (all resident layers).  Runs before the GPU is initialised: the workers
    are forked."""
    import multiprocessing as mp
    n = max(1, min(max_workers, len(os.sched_getaffinity(0)), w.batch))
    ctx = mp.get_context("fork")
    barrier, out = ctx.Barrier(n), ctx.Queue()
    procs = [ctx.Process(target=_oracle_share, args=(w, i, n, barrier, out)) for i in range(n)]
    for p in procs:
        p.start()
    res = [out.get() for _ in range(n + 1)]
    for p in procs:
        p.join()
        if p.exitcode != 0:
            raise RuntimeError(f"CPU oracle worker failed ({p.exitcode})")
    solo = [r for r in res if r[0] == "solo"][0]
    allr = [r for r in res if r[0] == "all"]
    live = sum(r[3] for r in allr)
    t_all = max(r[2] for r in allr) - min(r[1] for r in allr)     # one layer of the whole batch
    t_solo = (solo[2] - solo[1]) * n                               # the share alone, scaled to the batch
    step_all, step_solo = t_all * w.n_layers, t_solo * w.n_layers
    return {"value": round(live / step_all, 3), "unit": "query-tokens/s", "cores": n, "kind": "oracle",
            "single_thread_value": round(live / step_solo, 3),
            "host": {"nproc": os.cpu_count(), "usable_cpus": len(os.sched_getaffinity(0)), "cpu_model": cpu_model()},
            "sample": f"step 0 of {w.name}, layer 0 only (evict, embed, mask, attention over each query's "
                      f"history, advance; numpy float64): its {w.batch} slots dealt over {n} single-thread "
                      f"worker processes run together, {t_all:.2f} s wall; the first worker's share "
                      f"({len(range(0, w.batch, n))} slots) alone {solo[2] - solo[1]:.2f} s, x{n} for the "
                      f"single-thread figure; both x{w.n_layers} resident layers for the step.  Input "
                      f"generation and the initial batch's embedding are outside the timed part."}


def kernel_sources_sha256():
    """Hash of the decode attention's kernel sources and launch configuration:
    counters taken on other sources do not describe this kernel."""
    import hashlib
    h = hashlib.sha256()
    for f in ("common.hpp", "decode_attn.hpp", "decode_attn_mfma.hpp", "decode_launch.hpp"):
        with open(os.path.join(ROOT, "paper_2410_18701_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def copy_probe(nbytes, reps=5):
    """A plain device-to-device copy of nbytes (torch's copy kernel): the
    achievable HBM bandwidth on this GPU, and the reference kernel of known
    traffic for scaling rocprofv3's FETCH_SIZE / WRITE_SIZE counters."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    dst.copy_(src)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    t = a.elapsed_time(b) * 1e-3 / reps
    del src, dst
    return {"bytes_per_launch": 2 * nbytes, "avg_launch_us": round(t * 1e6, 2),
            "GB/s": round(2 * nbytes / t / 1e9, 1)}


def quantiles(xs):
    """Median and 90th percentile (nearest rank) of a list of timings."""
    ys = sorted(xs)
    if not ys:
        return None
    rank = lambda q: ys[min(len(ys) - 1, max(0, int(math.ceil(q * len(ys))) - 1))]
    return {"median": round(rank(0.5), 4), "p90": round(rank(0.9), 4), "n": len(ys)}


def read_probe(nbytes, reps=5, per_launch=False, n_bufs=1):
    """A read-only stream of nbytes (the workload library's reference kernel:
    64 KiB per workgroup, 16-byte non-temporal loads): what plain reads reach
    on this GPU, the practical ceiling of a read-dominated kernel such as
    decode attention.  per_launch: each launch timed between its own events
    (as the attention calls are), over n_bufs buffers in turn so that no
    launch finds its bytes in the last-level cache; otherwise reps launches
    back to back between two events."""
    import ctypes
    import torch
    from workload import gen
    lib = gen.dev_lib()
    nbytes = max(65536, nbytes // 65536 * 65536)
    bufs = [torch.empty(nbytes, dtype=torch.uint8, device="cuda") for _ in range(n_bufs)]
    for buf in bufs:
        buf.fill_(1)
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    launch = lambda i: lib.wl_device_read_stream(ctypes.c_void_p(bufs[i % n_bufs].data_ptr()), nbytes,
                                                 ctypes.c_void_p(flag.data_ptr()), stream)
    for i in range(n_bufs):
        if launch(i) != 0:
            raise RuntimeError("wl_device_read_stream failed")
    torch.cuda.synchronize()
    if per_launch:
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(reps)]
        for i, (a, b) in enumerate(evs):
            a.record()
            launch(i)
            b.record()
        torch.cuda.synchronize()
        t = sum(a.elapsed_time(b) for a, b in evs) * 1e-3 / reps
    else:
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for i in range(reps):
            launch(i)
        b.record()
        torch.cuda.synchronize()
        t = a.elapsed_time(b) * 1e-3 / reps
    del bufs, flag
    return {"bytes_per_launch": nbytes, "avg_launch_us": round(t * 1e6, 2), "GB/s": round(nbytes / t / 1e9, 1),
            "timing": "per launch" if per_launch else "back to back"}


def traffic_record(args, w):
    """The decode-attention traffic ratio measured with rocprofv3 on this
    workload, if it was taken on the current kernel sources."""
    name = TRAFFIC.get(w.name)
    if not name or args.split is not None:
        return None
    path = os.path.join(args.traffic_dir, name)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_sources_sha256") != kernel_sources_sha256() or "traffic_over_algorithmic" not in rec:
        return None
    return rec


def bench_decode(args, w, probes=True, no_scrub_steps=0):
    """The timed decode steps of workload w (its schedule's first warmup +
    steps steps, evictions scrubbing and releasing), then no_scrub_steps more
    whose evictions leave their tokens (kv_embed timed without placeholder
    writes).  Returns the result dict of the JSON line."""
    import torch

    from workload import driver

    copy_ref = copy_probe(args.copy_bytes) if probes and args.copy_bytes > 0 else None
    read_ref = read_probe(2 * args.copy_bytes) if probes and args.copy_bytes > 0 else None
    total_steps = args.warmup + args.steps
    log(f"{w.name}: building the initial batch ({w.n_layers} layers, {w.batch} slots)")
    cache, inputs = driver.open_cache(w, split=args.split)
    cap = cache.capacity

    def inputs_of(steps):
        need = sum(driver.prefill_bytes(w, n) for s in steps for n in w.steps[s].insert_lens)
        need += len(steps) * w.n_layers * w.batch * (w.n_q_heads + 2 * w.n_kv_heads) * w.head_dim * w.elem_bytes
        free, _ = torch.cuda.mem_get_info()
        if need + (2 << 30) > free:
            sys.exit(f"timed inputs need {need / 1e9:.1f} GB, {free / 1e9:.1f} GB free: use fewer --steps")
        out = []
        for s in steps:
            ev = w.steps[s]
            srcs = [inputs.prefill(q, n) for q, n in zip(ev.insert_qids, ev.insert_lens)]
            dec = [inputs.decode(s, layer) for layer in range(w.n_layers)]
            out.append((srcs, dec))
        return out

    for s in range(args.warmup):
        driver.run_step(cache, inputs, s, w.steps[s])
    torch.cuda.synchronize()

    log(f"{w.name}: {args.warmup} warmup steps done; generating the timed steps' inputs")
    pre = inputs_of(range(args.warmup, total_steps))
    mask_buf = torch.empty((w.batch, cap + 1), dtype=torch.uint8, device="cuda")
    ws = cache.workspace()
    outs = [torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=inputs.tdt, device="cuda")
            for _ in range(2)]
    torch.cuda.synchronize()

    def timed(steps, pre, scrub):
        """Runs the steps between events; every event exists (and has been
        recorded once) before the timed region starts, and the collector is
        off, so the host never stalls the stream."""
        n_ev = 2 * len(steps) * (3 + w.n_layers) + 2
        pool = [torch.cuda.Event(enable_timing=True) for _ in range(n_ev)]
        for e in pool:
            e.record()
        torch.cuda.synchronize()
        pool_it = iter(pool)
        E = lambda: next(pool_it)
        r = {"attn": [], "embed": [], "evict": [], "mask": [], "step": [],
             "bytes_attn": 0, "bytes_embed": 0, "bytes_evict": 0, "live": 0}
        gc.collect()
        gc.disable()
        t_start, t_end = E(), E()
        torch.cuda.synchronize()
        lead = queue_lead(args.lead_bytes)
        t_start.record()
        for i, s in enumerate(steps):
            ev = w.steps[s]
            srcs, dec = pre[i]
            _, _, lens = cache.query()
            a, b = E(), E()
            a.record()
            cache.evict(ev.evict, release=True, scrub=scrub)
            b.record()
            r["evict"].append((a, b))
            if scrub:
                r["bytes_evict"] += placeholder_bytes(w, lens, ev)
            if ev.insert:
                a, b = E(), E()
                a.record()
                cache.embed(ev.insert, ev.insert_lens, [x[0] for x in srcs], [x[1] for x in srcs])
                b.record()
                r["embed"].append((a, b))
                r["bytes_embed"] += embed_bytes(w, ev.insert_lens)
            a, b = E(), E()
            a.record()
            cache.build_mask(out=mask_buf)
            b.record()
            r["mask"].append((a, b))
            _, _, lens = cache.query()
            step_attn = attn_bytes(w, lens)
            for layer in range(w.n_layers):
                q, kn, vn = dec[layer]
                a, b = E(), E()
                a.record()
                cache.decode_attn(layer, q, kn, vn, out=outs[layer & 1])
                b.record()
                r["attn"].append((a, b))
                r["bytes_attn"] += step_attn
            r["step"].append((r["evict"][-1][0], r["attn"][-1][1]))
            r["live"] += sum(1 for n in lens if n > 0)
            cache.advance()
        t_end.record()
        torch.cuda.synchronize()
        del lead
        gc.enable()
        r["total_ms"] = t_start.elapsed_time(t_end)
        return r

    main = timed(range(args.warmup, total_steps), pre, scrub=True)
    log(f"{w.name}: {args.steps} timed steps done, {main['total_ms']:.1f} ms")
    del pre
    ms = lambda evs: sum(x.elapsed_time(y) for x, y in evs)
    attn_ms, embed_ms, evict_ms, mask_ms = ms(main["attn"]), ms(main["embed"]), ms(main["evict"]), ms(main["mask"])
    total_ms = main["total_ms"]
    n_attn = len(main["attn"])
    bytes_attn, bytes_embed, bytes_evict = main["bytes_attn"], main["bytes_embed"], main["bytes_evict"]
    attn_gbs = bytes_attn / (attn_ms * 1e-3) / 1e9
    embed_gbs = bytes_embed / (embed_ms * 1e-3) / 1e9 if embed_ms > 0 else None
    live_tokens = main["live"]
    value = live_tokens / (total_ms * 1e-3)

    rec = traffic_record(args, w)
    traffic = round(rec["traffic_over_algorithmic"] * bytes_attn / n_attn) if rec else None

    resident = ""
    if w.name == GQA_WORKLOAD:
        resident = (f" ({w.n_layers} of its {GQA_LAYERS} layers resident: the dense padded cache of all "
                    f"{GQA_LAYERS} exceeds HBM; each step decodes the {w.n_layers}, each at the real per-layer shape)")
    attn_kernel = "attn_mfma_kernel" if w.n_q_heads > w.n_kv_heads and w.dtype == "bf16" else "attn_kernel"
    result = {
        "metric": "decode-attention query-tokens/s + achieved HBM GB/s (attn, kv_embed) at 1 GPU",
        "value": round(value, 1),
        "unit": "query-tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(total_ms / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded counter-based generator, values ~N(0,1))",
        "config": {
            "workload": f"{w.name}{resident}: {w.dtype}, {w.n_layers} layers x {w.n_q_heads} q-heads / "
                        f"{w.n_kv_heads} kv-heads x head_dim {w.head_dim}, batch {w.batch}, "
                        f"initial padded length {w.L0}, ring capacity {cap}, "
                        f"{total_steps} decode steps with re-batching",
            "global_batch": w.batch, "seq_len": w.L0, "parallelism": "none (1 GPU)",
            "split_tokens": args.split,
        },
        "roofline": {
            "bound": "hbm", "kernel": f"decode_attn ({attn_kernel} + combine_kernel + the step's meta_kernel)",
            "achieved": round(attn_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(attn_gbs / PEAK_HBM_GBS, 4), "traffic": traffic,
            "bytes_per_launch": round(bytes_attn / n_attn), "avg_launch_us": round(attn_ms / n_attn * 1e3, 2),
        },
        "ops": {
            "decode_attn": {"ms_per_step": round(attn_ms / args.steps, 4), "GB/s": round(attn_gbs, 1),
                            "frac_of_peak": round(attn_gbs / PEAK_HBM_GBS, 4),
                            "query_tokens_per_s": round(live_tokens / (attn_ms * 1e-3), 1)},
            "kv_embed": {"ms_per_step": round(embed_ms / args.steps, 4),
                         "GB/s": round(embed_gbs, 1) if embed_gbs else None,
                         "frac_of_peak": round(embed_gbs / PEAK_HBM_GBS, 4) if embed_gbs else None,
                         "bytes_per_step": round(bytes_embed / args.steps),
                         "placeholder_bytes_per_step": round(bytes_evict / args.steps),
                         "GB/s_with_placeholders": round((bytes_embed + bytes_evict) / (embed_ms * 1e-3) / 1e9, 1)
                         if embed_ms > 0 else None,
                         "note": "evictions scrub (BATON_SCRUB): the placeholder writes they owe run in "
                                 "the same launch as the copy; GB/s counts the copied bytes only"},
            "kv_evict": {"ms_per_step": round(evict_ms / args.steps, 4)},
            "build_mask": {"ms_per_step": round(mask_ms / args.steps, 4)},
        },
        "per_step_ms": quantiles([x.elapsed_time(y) for x, y in main["step"]]),
        "decode_attn_call_us": quantiles([x.elapsed_time(y) * 1e3 for x, y in main["attn"]]),
        "timing": (f"HIP events on the launch stream; a {args.lead_bytes >> 20} MiB device copy queued just before "
                   "the timed region, outside it, keeps the host loop ahead of the GPU" if args.lead_bytes > 0
                   else "HIP events on the launch stream"),
    }
    if rec:
        result["roofline"]["traffic_over_algorithmic"] = rec["traffic_over_algorithmic"]
        result["roofline"]["traffic_source"] = "profiles/" + TRAFFIC[w.name]
    if w.name == GQA_WORKLOAD:
        # the same step with all 80 layers: attention and embedding scale with the layers
        layer_ms = (attn_ms + embed_ms) / args.steps
        ms80 = evict_ms / args.steps + mask_ms / args.steps + layer_ms * GQA_LAYERS / w.n_layers
        result["ops"]["estimate_80_layers"] = {
            "ms_per_step": round(ms80, 4), "query_tokens_per_s": round(live_tokens / args.steps / (ms80 * 1e-3), 1),
            "how": f"measured evict and mask per step, plus decode_attn and kv_embed per step x "
                   f"{GQA_LAYERS}/{w.n_layers} layers (a derived figure, not timed)"}

    if no_scrub_steps > 0:
        extra = range(total_steps, total_steps + no_scrub_steps)
        pre2 = inputs_of(extra)
        torch.cuda.synchronize()
        r2 = timed(extra, pre2, scrub=False)
        log(f"{w.name}: {no_scrub_steps} steps without scrubbing done")
        del pre2
        e_ms = ms(r2["embed"])
        result["ops"]["kv_embed_no_scrub"] = {
            "steps": no_scrub_steps, "ms_per_step": round(e_ms / no_scrub_steps, 4),
            "GB/s": round(r2["bytes_embed"] / (e_ms * 1e-3) / 1e9, 1) if e_ms > 0 else None,
            "frac_of_peak": round(r2["bytes_embed"] / (e_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4) if e_ms > 0 else None,
            "bytes_per_step": round(r2["bytes_embed"] / no_scrub_steps),
            "note": f"steps {extra.start}..{extra.stop - 1} after the timed ones, evictions without "
                    "BATON_SCRUB (the mask alone excludes the finished tokens): the launch copies only"}

    if probes and copy_ref:
        result["hbm_copy_reference"] = copy_ref
        result["hbm_read_reference"] = read_ref
        result["roofline"]["frac_of_read_reference"] = round(attn_gbs / read_ref["GB/s"], 4)
        # The same read at the attention's own bytes per call, each launch
        # timed alone as the calls are: what a single launch of that size
        # loses to filling and draining the GPU is in both.
        del cache, inputs, outs, ws, mask_buf
        gc.collect()
        torch.cuda.empty_cache()
        read_same = read_probe(round(bytes_attn / n_attn), reps=32, per_launch=True, n_bufs=4)
        result["hbm_read_reference_same_size"] = read_same
        result["roofline"]["frac_of_read_reference_same_size"] = round(attn_gbs / read_same["GB/s"], 4)
    return result


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (--gpus {args.gpus} requested); "
              "the batch shards by slot or by kv-head with no exchange on this path.", file=sys.stderr)
        sys.exit(2)

    from workload import configs

    total_steps = args.warmup + args.steps

    def workload(name, extra_steps=0):
        if name == GQA_WORKLOAD:
            return configs.gqa70b_b128_l8192(total_steps + extra_steps, n_layers=args.layers or GQA_RESIDENT)
        if args.layers:
            raise SystemExit(f"--layers applies to {GQA_WORKLOAD} only")
        return configs.CONFIGS[name](total_steps + extra_steps)

    plain = not args.no_pd and not args.model
    extra = args.no_scrub_steps if plain else 0
    w = workload(args.config, extra)
    # The CPU baseline first, while no GPU is initialised (its workers are forked).
    if plain and not args.no_cpu_baseline:
        log("CPU oracle baseline")
    cpu = cpu_baseline(w, args.cpu_workers) if plain and not args.no_cpu_baseline else None
    if cpu:
        log(f"CPU oracle baseline: {cpu['value']} query-tokens/s on {cpu['cores']} cores")

    import torch
    torch.cuda.set_device(0)
    if args.no_pd:
        print(json.dumps(bench_no_pd(args, w)), flush=True)
        return
    if args.model:
        print(json.dumps(bench_model(args, w)), flush=True)
        return
    result = bench_decode(args, w, probes=True, no_scrub_steps=extra)
    if not args.no_secondary and args.config == DEFAULT_WORKLOAD and args.split is None:
        gc.collect()
        torch.cuda.empty_cache()
        w2 = workload(SECONDARY_WORKLOAD)
        r2 = bench_decode(args, w2, probes=False)
        result["also"] = {SECONDARY_WORKLOAD: {
            "workload": r2["config"]["workload"], "value": r2["value"], "unit": r2["unit"],
            "ms_per_step": r2["ms_per_step"], "decode_attn": r2["ops"]["decode_attn"],
            "kv_embed": r2["ops"]["kv_embed"], "roofline": r2["roofline"],
            "per_step_ms": r2["per_step_ms"], "decode_attn_call_us": r2["decode_attn_call_us"]}}
    if cpu is not None:
        result["cpu_baseline"] = cpu
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
