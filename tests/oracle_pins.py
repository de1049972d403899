"""Pins of the CPU oracle: checks against what the paper and the mathematics fix.

Each pin takes the oracle module (so the mutation tests can hand it a copy with
one planted mistake) and raises AssertionError when the oracle disagrees.
"""
import itertools
import json
import math
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------- numbers --
def pin_widen_worked(O):
    """Stored bit patterns widened by hand.  bf16 (sign, 8 exponent bits, bias
    127, 7 mantissa bits): 0x3F80 = +2^0 x 1.0; 0xC020 = -2^1 x 1.25; 0x0001 is
    the smallest subnormal, 2^-126 x 2^-7; 0x0080 the smallest normal, 2^-126;
    0x7F7F the largest finite, 2^127 x (2 - 2^-7); 0x4049 = 2^1 x (1 + 73/128).
    fp32 the same with 23 mantissa bits."""
    inf = math.inf
    bf16 = [(0x3F80, 1.0), (0xC020, -2.5), (0x0001, 2.0 ** -133), (0x0080, 2.0 ** -126),
            (0x7F7F, (2.0 - 2.0 ** -7) * 2.0 ** 127), (0xFF80, -inf), (0x7F80, inf), (0x4049, 3.140625),
            (0x3F81, 1.0 + 2.0 ** -7), (0x3F7F, 1.0 - 2.0 ** -8), (0x8001, -(2.0 ** -133))]
    f32 = [(0x3F800000, 1.0), (0xC0200000, -2.5), (0x00000001, 2.0 ** -149), (0x00800000, 2.0 ** -126),
           (0x7F7FFFFF, (2.0 - 2.0 ** -23) * 2.0 ** 127), (0xFF800000, -inf), (0x3F800001, 1.0 + 2.0 ** -23)]
    for dtype, cases, st in ((O.BF16, bf16, np.uint16), (O.F32, f32, np.uint32)):
        got = O.widen(np.array([b for b, _ in cases], st), dtype)
        want = np.array([v for _, v in cases])
        assert np.array_equal(got, want), (dtype, got, want)
    # the sign of zero is kept, and NaN patterns stay NaN
    z = O.widen(np.array([0x8000, 0x0000], np.uint16), O.BF16)
    assert z[0] == 0.0 and math.copysign(1.0, z[0]) == -1.0 and math.copysign(1.0, z[1]) == 1.0
    assert np.all(np.isnan(O.widen(np.array([0x7FC0, 0xFFC1, 0x7F81], np.uint16), O.BF16)))


def pin_widen_exhaustive(O):
    """Every one of the 65,536 bf16 patterns against torch's bfloat16 type read
    as float64 (a library routine), and a sample of fp32 patterns against the
    C library's single-precision unpacking (struct)."""
    import struct

    import torch
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ref = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).double().numpy()
    got = O.widen(bits, O.BF16)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan]) and np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))
    rng = np.random.default_rng(17)
    words = np.concatenate([rng.integers(0, 1 << 32, 4096, dtype=np.uint64).astype(np.uint32),
                            np.array([0, 1, 0x7F7FFFFF, 0x80000000, 0x00800000, 0xFF800000], np.uint32)])
    ref32 = np.array([struct.unpack("<f", struct.pack("<I", int(u)))[0] for u in words])
    got32 = O.widen(words, O.F32)
    nan = np.isnan(ref32)
    assert np.array_equal(np.isnan(got32), nan) and np.array_equal(got32[~nan], ref32[~nan])


# ------------------------------------------------------------- attention --
def pin_attention_worked(O):
    """Hand-worked single-query cases (tests/golden/attention_worked.json, sec. 2.1)."""
    for c in _load("attention_worked.json")["cases"]:
        q = np.array(c["q"], float)
        K = np.array(c["K"], float)
        V = np.array(c["V"], float)
        scale = 1.0 / math.sqrt(len(q)) if c["scale"] is None else c["scale"]
        out = O.attend(q, K, V, scale)
        assert np.allclose(out, c["out"], rtol=0, atol=1e-12), (c["name"], out, c["out"])


def pin_attention_closed_forms(O):
    """Closed forms of softmax attention, on random inputs."""
    rng = np.random.default_rng(11)
    for n, D in ((1, 8), (2, 4), (17, 64), (300, 128)):
        q = rng.standard_normal(D)
        K = rng.standard_normal((n, D))
        V = rng.standard_normal((n, D))
        s = 1.0 / math.sqrt(D)
        # one token: the output is its value
        assert np.allclose(O.attend(q, K[:1], V[:1], s), V[0], atol=1e-14)
        # identical keys: uniform weights, the output is the mean value
        Krep = np.repeat(K[:1], n, axis=0)
        assert np.allclose(O.attend(q, Krep, V, s), V.mean(axis=0), atol=1e-12)
        # zero query: uniform weights
        assert np.allclose(O.attend(np.zeros(D), K, V, s), V.mean(axis=0), atol=1e-12)
        # identical values: the output is that value
        Vrep = np.repeat(V[:1], n, axis=0)
        assert np.allclose(O.attend(q, K, Vrep, s), V[0], atol=1e-12)
        # two tokens: o = v0 + sigmoid(s1 - s0) (v1 - v0)
        if n >= 2:
            d = s * (K[1] @ q - K[0] @ q)
            want = V[0] + (V[1] - V[0]) / (1.0 + math.exp(-d))
            assert np.allclose(O.attend(q, K[:2], V[:2], s), want, atol=1e-12)


def pin_attention_sdpa(O):
    """The library routine: torch's scaled_dot_product_attention on the CPU in float64."""
    import torch
    import torch.nn.functional as F
    rng = np.random.default_rng(5)
    for n, D, scale in ((1, 64, None), (5, 64, None), (129, 128, None), (40, 32, 0.3)):
        q = rng.standard_normal(D)
        K = rng.standard_normal((n, D))
        V = rng.standard_normal((n, D))
        s = 1.0 / math.sqrt(D) if scale is None else scale
        ref = F.scaled_dot_product_attention(
            torch.tensor(q)[None, None, None], torch.tensor(K)[None, None],
            torch.tensor(V)[None, None], scale=scale).numpy()[0, 0, 0]
        assert np.allclose(O.attend(q, K, V, s), ref, atol=1e-12), (n, D)


def pin_attention_permutation(O):
    """Attention is a set function of the (key, value) pairs."""
    rng = np.random.default_rng(3)
    q = rng.standard_normal(16)
    K = rng.standard_normal((9, 16))
    V = rng.standard_normal((9, 16))
    p = rng.permutation(9)
    assert np.allclose(O.attend(q, K, V, 0.25), O.attend(q, K[p], V[p], 0.25), atol=1e-13)


# ----------------------------------------------------- the padded batch --
def _code(qid, t):
    return float(1000 * qid + t + 1)


def _decode_cell(x):
    if math.isinf(x):
        return "."
    c = int(x) - 1
    return f"q{c // 1000}.{c % 1000}"


def _src(qid, n):
    """fp32 bits [1 layer][1 head][n][1 dim] whose values name (qid, t)."""
    vals = np.array([_code(qid, t) for t in range(n)], np.float32).reshape(1, 1, n, 1)
    return vals.view(np.uint32)


def pin_insertion_replay(O):
    """Replay of the sec. 4.1 / sec. 4.2 insertion story against hand-derived states
    (tests/golden/insertion_replay.json): lengths, cell contents, mask."""
    g = _load("insertion_replay.json")
    B = g["batch"]
    pb = O.PaddedBatch(1, B, 1, 1, 1, O.F32)
    slot_qid = [None] * B
    for op in g["ops"]:
        if op["op"] == "embed":
            srcs = [_src(q, n) for q, n in zip(op["qids"], op["lens"])]
            pb.embed(op["slots"], op["lens"], srcs, srcs)
            for s, q in zip(op["slots"], op["qids"]):
                slot_qid[s] = q
        elif op["op"] == "evict":
            pb.evict(op["slots"], release=True)
            for s in op["slots"]:
                slot_qid[s] = None
        elif op["op"] == "decode":
            kn = np.full((B, 1, 1), O.NEG_INF_BITS[O.F32], np.uint32)
            for b in range(B):
                if slot_qid[b] is not None:
                    kn[b, 0, 0] = np.float32(_code(slot_qid[b], pb.lens[b])).view(np.uint32)
            q = np.zeros((B, 1, 1), np.uint32)
            pb.decode_layer(0, q, kn, kn)
            pb.advance()
        assert pb.L == op["L"], (op, pb.L)
        cells = pb.K[0, :, 0, :, 0].view(np.float32)
        for b in range(B):
            got = " ".join(_decode_cell(x) for x in cells[b])
            assert got == op["rows"][b], (op["op"], b, got, op["rows"][b])
        want_mask = np.array([[int(x) for x in r.split()] for r in op["mask"]], np.uint8)
        assert np.array_equal(pb.mask(), want_mask), (op["op"], pb.mask(), want_mask)


def pin_gqa_mapping(O):
    """Grouped-query reading (tests/golden/attention_worked.json, gqa)."""
    g = _load("attention_worked.json")["gqa"]
    Hq, Hkv, D = g["n_q_heads"], g["n_kv_heads"], 4
    pb = O.PaddedBatch(1, 1, Hq, Hkv, D, O.F32)
    rng = np.random.default_rng(0)
    n = 6
    k = rng.standard_normal((1, Hkv, n, D)).astype(np.float32).view(np.uint32)
    v = np.stack([np.full((n, D), c, np.float32) for c in g["v_const"]])[None].view(np.uint32)
    pb.embed([0], [n], [k], [v])
    q = rng.standard_normal((1, Hq, D)).astype(np.float32).view(np.uint32)
    kn = rng.standard_normal((1, Hkv, D)).astype(np.float32).view(np.uint32)
    vn = np.array([[np.full(D, c, np.float32) for c in g["v_const"]]]).view(np.uint32)
    out = pb.decode_layer(0, q, kn, vn)
    assert np.allclose(out[0], np.array(g["out_const"])[:, None], atol=1e-12), out


def _random_ops(rng, B, steps, max_len):
    ops = []
    live = set()
    for _ in range(steps):
        free = [b for b in range(B) if b not in live]
        r = rng.random()
        if live and r < 0.3:
            k = int(rng.integers(1, len(live) + 1))
            ev = sorted(rng.choice(sorted(live), k, replace=False).tolist())
            ops.append(("evict", ev))
            live -= set(ev)
        elif free and r < 0.6:
            k = int(rng.integers(1, len(free) + 1))
            ins = rng.choice(free, k, replace=False).tolist()
            ops.append(("embed", ins, [int(rng.integers(1, max_len + 1)) for _ in ins]))
            live |= set(ins)
        else:
            ops.append(("decode",))
    return ops


def _run(O, ops, NL, B, Hq, Hkv, D, dtype, seed, fill=None, check=None):
    """Apply ops to a PaddedBatch with random tensors; call check(pb, op, outs)."""
    rng = np.random.default_rng(seed)
    pb = O.PaddedBatch(NL, B, Hq, Hkv, D, dtype, fill_bits=fill)

    def rand_bits(shape):
        x = rng.standard_normal(shape).astype(np.float32)
        if dtype == O.BF16:
            return (x.view(np.uint32) >> 16).astype(np.uint16)
        return x.view(np.uint32)

    for op in ops:
        outs = None
        if op[0] == "evict":
            pb.evict(op[1], release=True)
        elif op[0] == "embed":
            ks = [rand_bits((NL, Hkv, n, D)) for n in op[2]]
            vs = [rand_bits((NL, Hkv, n, D)) for n in op[2]]
            pb.embed(op[1], op[2], ks, vs)
        else:
            outs = []
            for layer in range(NL):
                q = rand_bits((B, Hq, D))
                kn = rand_bits((B, Hkv, D))
                vn = rand_bits((B, Hkv, D))
                o = pb.decode_layer(layer, q, kn, vn)
                outs.append((q, o, pb.decode_layer_padded(layer, q)))
            pb.advance()
        if check is not None:
            check(pb, op, outs)
    return pb


def pin_isolation_invariant(O):
    """The paper's correctness claim (sec. 4.1): a query's output in the shaped,
    masked batch equals its output over its own tokens alone."""
    rng = np.random.default_rng(21)

    def check(pb, op, outs):
        if outs:
            for _, iso, batched in outs:
                assert np.allclose(iso, batched, rtol=0, atol=1e-12)

    for trial in range(6):
        ops = _random_ops(rng, B=4, steps=14, max_len=9)
        _run(O, ops, 2, 4, 4, 2, 8, O.BF16 if trial % 2 else O.F32, seed=trial, check=check)


def pin_layout_invariants(O):
    """Shape rules of secs. 4.1-4.2 on random op sequences: live rows are
    placeholders then the query's own history (end-aligned), free rows are all
    placeholders, L is the longest live row after a release, an insertion makes
    L = max(L, l_q), the mask row is a suffix of ones of length len+1."""
    rng = np.random.default_rng(8)

    def check(pb, op, outs):
        fill = pb.fill
        for b in range(pb.B):
            n = pb.lens[b]
            assert 0 <= n <= pb.L
            row = pb.K[:, b]
            if n == 0:
                assert np.all(row == fill)
            else:
                assert np.all(row[:, :, : pb.L - n] == fill)
                assert np.array_equal(row[:, :, pb.L - n:], pb.hist_k[b])
                assert np.array_equal(pb.V[:, b, :, pb.L - n:], pb.hist_v[b])
            m = pb.mask()[b]
            want = np.zeros(pb.L + 1, np.uint8)
            if n:
                want[pb.L - n:] = 1
            assert np.array_equal(m, want)
        # the mask the batch built step by step is the closed form of its lengths
        assert np.array_equal(pb.mask(), O.build_mask(pb.L, pb.lens))
        if op[0] == "evict":
            assert pb.L == max(pb.lens)
        elif op[0] == "embed":
            assert pb.L == max(check.prev_L, max(op[2]))
        else:
            assert pb.L == check.prev_L + 1
        check.prev_L = pb.L

    for trial in range(8):
        check.prev_L = 0
        ops = _random_ops(rng, B=3, steps=16, max_len=7)
        _run(O, ops, 1, 3, 2, 1, 4, O.F32, seed=100 + trial, check=check)


def pin_embed_order_and_release(O):
    """Insertions commute (one growth to the longest equals growths one by one),
    and releasing twice drops nothing more."""
    rng = np.random.default_rng(4)
    for trial in range(10):
        lens = [int(x) for x in rng.integers(1, 12, size=3)]
        base = int(rng.integers(1, 12))
        srcs = [rng.integers(0, 2**31, size=(1, 2, n, 3)).astype(np.uint32) for n in [base] + lens]
        states = []
        for order in itertools.permutations(range(3)):
            pb = O.PaddedBatch(1, 4, 2, 2, 3, O.F32)
            pb.embed([0], [base], [srcs[0]], [srcs[0]])
            pb.embed([1 + i for i in order], [lens[i] for i in order],
                     [srcs[1 + i] for i in order], [srcs[1 + i] for i in order])
            states.append((pb.L, pb.K.copy(), pb.mask()))
        for L, K, M in states[1:]:
            assert L == states[0][0] and np.array_equal(K, states[0][1])
            assert np.array_equal(M, states[0][2])
        assert states[0][0] == max([base] + lens)
        pb.evict([0], release=True)
        L1 = pb.L
        assert pb.release() == 0 and pb.L == L1


def pin_brute_force_small(O):
    """Every sequence of up to four operations on 2 slots with lengths <= 2:
    the padded rows always equal placeholders + the query's own history, and
    every query's batched output equals its isolated output."""
    B = 2
    choices = []
    for s in range(B):
        for n in (1, 2):
            choices.append(("embed", [s], [n]))
        choices.append(("evict", [s]))
    choices.append(("evict", [0, 1]))
    choices.append(("embed", [0, 1], [2, 1]))
    choices.append(("decode",))
    count = 0

    def check(pb, op, outs):
        for b in range(pb.B):
            n = pb.lens[b]
            if n:
                assert np.array_equal(pb.K[:, b, :, pb.L - n:], pb.hist_k[b])
                assert np.all(pb.K[:, b, :, : pb.L - n] == pb.fill)
            else:
                assert np.all(pb.K[:, b] == pb.fill)
        if outs:
            for _, iso, batched in outs:
                assert np.allclose(iso, batched, atol=1e-12)

    for length in range(1, 5):
        for seq in itertools.product(choices, repeat=length):
            live = set()
            ok = True
            for op in seq:      # keep only valid sequences
                if op[0] == "embed":
                    ok &= not (set(op[1]) & live)
                    live |= set(op[1])
                elif op[0] == "evict":
                    ok &= set(op[1]) <= live
                    live -= set(op[1])
            if not ok:
                continue
            _run(O, list(seq), 1, B, 2, 1, 2, O.F32, seed=length, check=check)
            count += 1
    assert count > 100


def pin_placeholder_poison(O):
    """Placeholder bits never enter the arithmetic: -inf, 0 and NaN placeholders
    give bit-identical outputs (the paper's -inf would poison a product with 0)."""
    rng = np.random.default_rng(9)
    ops = _random_ops(rng, B=3, steps=12, max_len=6)
    results = []
    for fill in (0xFF800000, 0x00000000, 0x7FC00001):
        outs = []
        _run(O, ops, 1, 3, 2, 2, 4, O.F32, seed=77, fill=fill,
             check=lambda pb, op, o: outs.extend(x[1] for x in (o or [])))
        results.append(outs)
    for other in results[1:]:
        assert len(other) == len(results[0])
        for a, b in zip(results[0], other):
            assert np.array_equal(a, b)
            assert np.all(np.isfinite(a))


def pin_error_paths(O):
    """Invalid operations are refused and leave the batch as it was."""
    pb = O.PaddedBatch(1, 3, 1, 1, 2, O.F32)
    src = np.zeros((1, 1, 4, 2), np.uint32)
    pb.embed([0], [4], [src], [src])
    before = (pb.L, list(pb.lens), pb.K.copy())
    for bad in (lambda: pb.evict([1]), lambda: pb.embed([0], [2], [src[:, :, :2]], [src[:, :, :2]]),
                lambda: pb.embed([1, 1], [1, 1], [src[:, :, :1]] * 2, [src[:, :, :1]] * 2),
                lambda: pb.embed([2], [0], [src[:, :, :0]], [src[:, :, :0]]),
                lambda: pb.evict([5]), lambda: pb.advance()):
        try:
            bad()
        except (ValueError, LookupError, RuntimeError):
            pass
        else:
            raise AssertionError("invalid operation accepted")
        assert (pb.L, list(pb.lens)) == before[:2] and np.array_equal(pb.K, before[2])


ALL_PINS = [pin_widen_worked, pin_widen_exhaustive, pin_attention_worked, pin_attention_closed_forms, pin_attention_sdpa,
            pin_attention_permutation, pin_insertion_replay, pin_gqa_mapping,
            pin_isolation_invariant, pin_layout_invariants, pin_embed_order_and_release,
            pin_brute_force_small, pin_placeholder_poison, pin_error_paths]


def pin_preemption_round_trip(O):
    """Sec. 4.3 preemption: a query stored aside (extract), evicted, and embedded
    again into another slot later computes what it would have computed in place:
    same inputs, bit-identical output; and what extract returns is its own history."""
    import copy
    rng = np.random.default_rng(31)
    NL, B, Hq, Hkv, D = 2, 4, 4, 2, 8

    def bits(shape):
        return rng.standard_normal(shape).astype(np.float32).view(np.uint32)

    pb = O.PaddedBatch(NL, B, Hq, Hkv, D, O.F32)
    lens = [5, 9, 3]
    pb.embed([0, 1, 2], lens, [bits((NL, Hkv, n, D)) for n in lens], [bits((NL, Hkv, n, D)) for n in lens])
    for _ in range(2):
        for layer in range(NL):
            pb.decode_layer(layer, bits((B, Hq, D)), bits((B, Hkv, D)), bits((B, Hkv, D)))
        pb.advance()
    q, kn, vn = bits((B, Hq, D)), bits((B, Hkv, D)), bits((B, Hkv, D))
    stay = copy.deepcopy(pb)
    want = stay.decode_layer(0, q, kn, vn)[1]
    (k1, v1), = pb.extract([1])
    assert np.array_equal(k1, pb.hist_k[1]) and np.array_equal(v1, pb.hist_v[1])
    pb.evict([1], release=True)
    pb.embed([3], [k1.shape[2]], [k1], [v1])
    q2, kn2, vn2 = q.copy(), kn.copy(), vn.copy()
    q2[3], kn2[3], vn2[3] = q[1], kn[1], vn[1]
    got = pb.decode_layer(0, q2, kn2, vn2)[3]
    assert np.array_equal(got, want)


ALL_PINS.append(pin_preemption_round_trip)


# ------------------------------------- in-batch prefill (no P&D separation) --
_PAD_CODE = 999999.0


def pin_inbatch_prefill_replay(O):
    """Replay of the sec. 4.1 insertion story without prefill/decode separation
    against hand-derived states (tests/golden/inbatch_prefill_replay.json): L,
    cells (holes included), masks (the l_am + l_q - 1 wide mask of a prefill
    step), and the outputs of zero queries (means of the attended values)."""
    g = _load("inbatch_prefill_replay.json")
    B = g["batch"]
    pb = O.PaddedBatch(1, B, 1, 1, 1, O.F32)
    slot_qid = [None] * B
    count = [0] * B          # tokens in each query's own history
    for op in g["ops"]:
        if op["op"] == "embed":
            srcs = [_src(q, n) for q, n in zip(op["qids"], op["lens"])]
            pb.embed(op["slots"], op["lens"], srcs, srcs)
            for s, q, n in zip(op["slots"], op["qids"], op["lens"]):
                slot_qid[s], count[s] = q, n
        elif op["op"] == "evict":
            pb.evict(op["slots"], release=True)
            for s in op["slots"]:
                slot_qid[s], count[s] = None, 0
        elif op["op"] == "shape":
            l_am = pb.L + 1
            pb.shape_insert(op["slots"], op["lens"])
            shaped = {s: (q, n) for s, q, n in zip(op["slots"], op["qids"], op["lens"])}
            assert pb.mask().shape[1] == l_am + max(op["lens"]) - 1
        elif op["op"] == "step":
            T = pb.step_width()
            pending = pb._shape or {}
            kn = np.full((B, T, 1, 1), _PAD_CODE, np.float32)
            for b in range(B):
                if b in pending:
                    q, n = shaped[b]
                    for p in range(n):
                        kn[b, T - n + p] = _code(q, p)
                elif slot_qid[b] is not None:
                    kn[b, 0] = _code(slot_qid[b], count[b])
            kn = kn.view(np.uint32)
            q0 = np.zeros((B, T, 1, 1), np.uint32)
            if pending:
                out = pb.decode_layer(0, q0, kn, kn)
            else:
                out = pb.decode_layer(0, q0[:, 0], kn[:, 0], kn[:, 0])[:, None]
            for b in range(B):
                for t in range(T):
                    want = op["out"][b][t]
                    got = out[b, t, 0, 0]
                    if want is None:
                        assert math.isnan(got), (op, b, t, got)
                    else:
                        assert abs(got - want) < 1e-9, (op, b, t, got, want)
            pb.advance()
            for b in range(B):
                if b in pending:
                    slot_qid[b], count[b] = shaped[b][0], shaped[b][1]
                elif slot_qid[b] is not None:
                    count[b] += 1
        assert pb.L == op["L"], (op, pb.L)
        cells = pb.K[0, :, 0, :, 0].view(np.float32)
        for b in range(B):
            got = " ".join(_decode_cell(x) for x in cells[b])
            assert got == op["rows"][b], (op["op"], b, got, op["rows"][b])
        want_mask = np.array([[int(x) for x in r.split()] for r in op["mask"]], np.uint8)
        assert np.array_equal(pb.mask(), want_mask), (op["op"], pb.mask(), want_mask)


def pin_inbatch_prefill_sdpa(O):
    """The new query's outputs in a prefill step are causal self-attention over
    its prompt: torch's scaled_dot_product_attention(is_causal=True) in float64
    on the CPU, per q-head with the grouped kv-head; and its cached keys/values
    afterwards are exactly its prompt's."""
    import torch
    import torch.nn.functional as F
    rng = np.random.default_rng(41)
    NL, B, Hq, Hkv, D = 1, 3, 4, 2, 16

    def bits(shape):
        return rng.standard_normal(shape).astype(np.float32).view(np.uint32)

    pb = O.PaddedBatch(NL, B, Hq, Hkv, D, O.F32)
    pb.embed([0, 2], [5, 3], [bits((NL, Hkv, 5, D)), bits((NL, Hkv, 3, D))],
             [bits((NL, Hkv, 5, D)), bits((NL, Hkv, 3, D))])
    l_new = 7
    pb.shape_insert([1], [l_new])
    T = pb.step_width()
    q, kn, vn = bits((B, T, Hq, D)), bits((B, T, Hkv, D)), bits((B, T, Hkv, D))
    out = pb.decode_layer(0, q, kn, vn)
    g = Hq // Hkv
    for hq in range(Hq):
        h = hq // g
        Q = torch.tensor(O.widen(q[1, :, hq], O.F32))[None, None]
        K = torch.tensor(O.widen(kn[1, :, h], O.F32))[None, None]
        V = torch.tensor(O.widen(vn[1, :, h], O.F32))[None, None]
        ref = F.scaled_dot_product_attention(Q, K, V, is_causal=True).numpy()[0, 0]
        assert np.allclose(out[1, :, hq], ref, rtol=0, atol=1e-12), hq
    pb.advance()
    assert np.array_equal(pb.K[0, 1][:, pb.L - l_new:], kn[1].transpose(1, 0, 2))
    assert np.array_equal(pb.hist_v[1][0], vn[1].transpose(1, 0, 2))


def _random_ops_shaped(rng, B, steps, max_len):
    """Random sequences that also prefill new queries inside the batch."""
    ops = []
    live = set()
    for _ in range(steps):
        free = [b for b in range(B) if b not in live]
        r = rng.random()
        if live and r < 0.25:
            k = int(rng.integers(1, len(live) + 1))
            ev = sorted(rng.choice(sorted(live), k, replace=False).tolist())
            ops.append(("evict", ev))
            live -= set(ev)
        elif free and r < 0.45:
            k = int(rng.integers(1, len(free) + 1))
            ins = rng.choice(free, k, replace=False).tolist()
            ops.append(("embed", ins, [int(rng.integers(1, max_len + 1)) for _ in ins]))
            live |= set(ins)
        elif free and r < 0.7:
            k = int(rng.integers(1, len(free) + 1))
            ins = rng.choice(free, k, replace=False).tolist()
            ops.append(("shape", ins, [int(rng.integers(1, max_len + 1)) for _ in ins]))
            live |= set(ins)
        else:
            ops.append(("decode",))
    return ops


def _run_shaped(O, ops, NL, B, Hq, Hkv, D, dtype, seed, fill=None, check=None):
    """Like _run; a ("shape", slots, lens) op registers the prefill and runs its step."""
    rng = np.random.default_rng(seed)
    pb = O.PaddedBatch(NL, B, Hq, Hkv, D, dtype, fill_bits=fill)

    def rand_bits(shape):
        x = rng.standard_normal(shape).astype(np.float32)
        if dtype == O.BF16:
            return (x.view(np.uint32) >> 16).astype(np.uint16)
        return x.view(np.uint32)

    for op in ops:
        outs = None
        if op[0] == "evict":
            pb.evict(op[1], release=True)
        elif op[0] == "embed":
            ks = [rand_bits((NL, Hkv, n, D)) for n in op[2]]
            vs = [rand_bits((NL, Hkv, n, D)) for n in op[2]]
            pb.embed(op[1], op[2], ks, vs)
        else:
            if op[0] == "shape":
                pb.shape_insert(op[1], op[2])
            T = pb.step_width()
            pre = (B, T) if op[0] == "shape" else (B,)
            outs = []
            for layer in range(NL):
                q = rand_bits(pre + (Hq, D))
                kn = rand_bits(pre + (Hkv, D))
                vn = rand_bits(pre + (Hkv, D))
                o = pb.decode_layer(layer, q, kn, vn)
                outs.append((q, o, pb.decode_layer_padded(layer, q)))
            pb.advance()
        if check is not None:
            check(pb, op, outs)
    return pb


def pin_inbatch_prefill_isolation(O):
    """Sec. 4.1's correctness claim with prefills inside the batch: every query's
    output over the holey, masked rows equals its output over its own tokens
    (the new query's: causal over its prompt), and positions without a token
    are the same ones in both; rows are placeholders except where the mask is 1,
    where they hold the query's own history in order; the mask has L + 1
    columns and a row's span reaches its first token."""
    rng = np.random.default_rng(43)

    def check(pb, op, outs):
        for _, iso, batched in outs or []:
            assert np.array_equal(np.isnan(iso), np.isnan(batched))
            assert np.allclose(np.nan_to_num(iso), np.nan_to_num(batched), rtol=0, atol=1e-12)
        M = pb.mask()
        assert M.shape == (pb.B, pb.L + 1)
        for b in range(pb.B):
            live = pb.lens[b] > 0
            assert M[b, pb.L] == (1 if live else 0)
            ones = np.flatnonzero(M[b, :pb.L])
            if not live:
                assert len(ones) == 0 and np.all(pb.K[:, b] == pb.fill)
                continue
            assert ones[0] == pb.L - pb.lens[b]
            want = np.stack([np.stack([O.expected_row_masked(M[b, :pb.L], pb.hist_k[b][l, h], pb.fill, pb.dtype)
                                       for h in range(pb.Hkv)]) for l in range(pb.NL)])
            assert np.array_equal(pb.K[:, b], want)

    for trial in range(6):
        ops = _random_ops_shaped(rng, B=4, steps=14, max_len=6)
        _run_shaped(O, ops, 2, 4, 4, 2, 8, O.BF16 if trial % 2 else O.F32, seed=200 + trial, check=check)


ALL_PINS += [pin_inbatch_prefill_replay, pin_inbatch_prefill_sdpa, pin_inbatch_prefill_isolation]


def pin_move_is_a_permutation(O):
    """Moving queries between slots (sec. 4.3) permutes the batch and nothing
    else: after a move the batch equals the batch that had the queries in the
    new slots from the start -- rows, mask, lengths, and every later output."""
    rng = np.random.default_rng(51)
    NL, B, Hq, Hkv, D = 2, 5, 4, 2, 8

    def bits(shape):
        return rng.standard_normal(shape).astype(np.float32).view(np.uint32)

    lens = [6, 3, 9]
    ks = [bits((NL, Hkv, n, D)) for n in lens]
    vs = [bits((NL, Hkv, n, D)) for n in lens]
    a = O.PaddedBatch(NL, B, Hq, Hkv, D, O.F32)
    a.embed([1, 3, 4], lens, ks, vs)
    a.move([3, 4], [0, 2])                       # compact: live rows 0, 1, 2
    b = O.PaddedBatch(NL, B, Hq, Hkv, D, O.F32)
    b.embed([1, 0, 2], lens, ks, vs)
    assert a.L == b.L and a.lens == b.lens
    assert np.array_equal(a.K, b.K) and np.array_equal(a.V, b.V) and np.array_equal(a.mask(), b.mask())
    for _ in range(2):
        for layer in range(NL):
            q, kn, vn = bits((B, Hq, D)), bits((B, Hkv, D)), bits((B, Hkv, D))
            assert np.array_equal(a.decode_layer(layer, q, kn, vn), b.decode_layer(layer, q, kn, vn))
        a.advance()
        b.advance()
    try:
        a.move([0], [1])
    except LookupError:
        pass
    else:
        raise AssertionError("moved into a live slot")


ALL_PINS.append(pin_move_is_a_permutation)
