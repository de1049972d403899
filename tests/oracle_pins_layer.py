"""Pins of the decode-layer oracle (oracle/llama_layer.py): checks against
closed forms, independent formulations and library routines.  Each pin takes
the oracle module so that the mutation tests can hand it a planted mistake."""
import math

import numpy as np


def pin_rmsnorm(L):
    """torch's rms_norm in float64; mean square of the output with unit gain is
    ms / (ms + eps); zero eps makes it scale-invariant."""
    import torch
    import torch.nn.functional as F
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 64)) * 3.0
    g = rng.standard_normal(64)
    ref = F.rms_norm(torch.tensor(x), (64,), torch.tensor(g), eps=1e-5).numpy()
    assert np.allclose(L.rmsnorm(x, g, 1e-5), ref, rtol=0, atol=1e-12)
    y = L.rmsnorm(x, np.ones(64), 1e-5)
    ms = np.mean(x * x, axis=-1)
    assert np.allclose(np.mean(y * y, axis=-1), ms / (ms + 1e-5), rtol=1e-12)
    assert np.allclose(L.rmsnorm(7.5 * x, g, 0.0), L.rmsnorm(x, g, 0.0), atol=1e-12)


def pin_rope(L):
    """Rotary embedding against the complex-number form (pair i as a + ib times
    e^{i pos theta^(-2i/D)}); norms of pairs kept; position 0 is the identity;
    dot products depend on the position difference only."""
    rng = np.random.default_rng(2)
    D, theta = 16, 10000.0
    v = rng.standard_normal((3, D))
    pos = np.array([0.0, 5.0, 1234.0])
    got = L.rope(v, pos, theta)
    z = v[:, :D // 2] + 1j * v[:, D // 2:]
    ang = pos[:, None] * theta ** (-np.arange(D // 2) * 2.0 / D)
    zr = z * np.exp(1j * ang)
    assert np.allclose(got, np.concatenate([zr.real, zr.imag], axis=-1), rtol=0, atol=1e-12)
    assert np.allclose(got[0], v[0], atol=0)
    pair = lambda u: u[..., :D // 2] ** 2 + u[..., D // 2:] ** 2
    assert np.allclose(pair(got), pair(v), rtol=1e-12)
    q, k = rng.standard_normal(D), rng.standard_normal(D)
    for m, n, s in ((3, 1, 10), (100, 250, 7), (0, 9, 1000)):
        a = L.rope(q, m, theta) @ L.rope(k, n, theta)
        b = L.rope(q, m + s, theta) @ L.rope(k, n + s, theta)
        assert abs(a - b) < 1e-9, (m, n, s, a, b)
    # D = 2: a plain rotation by pos radians
    u = np.array([1.0, 0.0])
    assert np.allclose(L.rope(u, 0.5, theta), [math.cos(0.5), math.sin(0.5)], atol=1e-15)


def pin_silu(L):
    """torch's silu; silu(0) = 0; silu(z) - silu(-z) = z."""
    import torch
    import torch.nn.functional as F
    z = np.linspace(-20, 20, 401)
    assert np.allclose(L.silu(z), F.silu(torch.tensor(z)).numpy(), rtol=0, atol=1e-12)
    assert L.silu(np.array([0.0]))[0] == 0.0
    assert np.allclose(L.silu(z) - L.silu(-z), z, atol=1e-12)


def pin_linear_and_split(L):
    """A worked product (weights stored [out][in]) and the fused projection's
    layout: q rows, then k, then v."""
    x = np.array([[1.0, 2.0, 3.0]])
    w = np.array([[1.0, 0.0, -1.0], [2.0, 1.0, 0.0]])
    assert np.array_equal(L.linear(x, w), np.array([[-2.0, 4.0]]))
    Hq, Hkv, D = 4, 2, 3
    qkv = np.arange((Hq + 2 * Hkv) * D, dtype=np.float64)[None]
    q, k, v = L.split_qkv(qkv, Hq, Hkv, D)
    assert q[0, 1, 0] == 3 and k[0, 0, 0] == Hq * D and v[0, 1, 2] == (Hq + Hkv) * D + D + 2


def pin_to_bits(L):
    """Round-to-nearest-even into bf16: ties go to the even mantissa."""
    vals = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1.0 + 2 ** -7])
    want = np.array([0x3F80, 0x3F80, 0x3F82, 0xC020, 0x3F81], np.uint16)
    assert np.array_equal(L.to_bits(vals, L.BF16), want)


def _batch(O, rng, NL, B, Hq, Hkv, D, lens):
    pb = O.PaddedBatch(NL, B, Hq, Hkv, D, O.F32)
    bits = lambda shape: rng.standard_normal(shape).astype(np.float32).view(np.uint32)
    pb.embed(list(range(len(lens))), lens, [bits((NL, Hkv, n, D)) for n in lens],
             [bits((NL, Hkv, n, D)) for n in lens])
    return pb


def pin_layer_residual(L):
    """The layer adds its two blocks to the residual stream: with the output and
    down projections zero the stream is unchanged; with the down projection zero
    and an identity output projection it gains exactly the attention output."""
    import oracle.baton_oracle as O
    rng = np.random.default_rng(3)
    Hq, Hkv, D, hid, F = 4, 2, 8, 32, 16
    w = {"norm1": rng.standard_normal(hid), "qkv": rng.standard_normal(((Hq + 2 * Hkv) * D, hid)) / 6,
         "o": np.zeros((hid, hid)), "norm2": rng.standard_normal(hid),
         "gate_up": rng.standard_normal((2 * F, hid)) / 6, "down": np.zeros((hid, F))}
    x = rng.standard_normal((3, hid))
    pb = _batch(O, rng, 1, 3, Hq, Hkv, D, [4, 7, 2])
    out = L.decode_layer(pb, 0, x, w, [4, 7, 2], 10000.0, 1e-5)
    assert np.array_equal(out, x)
    w["o"] = np.eye(hid)
    pb2 = _batch(O, np.random.default_rng(3), 1, 3, Hq, Hkv, D, [4, 7, 2])
    # the same attention, recomputed independently from the layer's own q/k/v
    h = L.rmsnorm(x, w["norm1"], 1e-5)
    q, k, v = L.split_qkv(L.linear(h, w["qkv"]), Hq, Hkv, D)
    pos = np.array([4.0, 7.0, 2.0])[:, None]
    qb, kb, vb = (L.to_bits(L.rope(q, pos, 1e4), O.F32), L.to_bits(L.rope(k, pos, 1e4), O.F32),
                  L.to_bits(v, O.F32))
    att = np.zeros((3, Hq, D))
    for b in range(3):
        for hq in range(Hq):
            hh = hq // (Hq // Hkv)
            K = O.widen(np.concatenate([pb2.hist_k[b][0, hh], kb[b, hh][None]]), O.F32)
            V = O.widen(np.concatenate([pb2.hist_v[b][0, hh], vb[b, hh][None]]), O.F32)
            att[b, hq] = O.attend(O.widen(qb[b, hq], O.F32), K, V, 1 / math.sqrt(D))
    out2 = L.decode_layer(pb2, 0, x, w, [4, 7, 2], 10000.0, 1e-5)
    assert np.allclose(out2, x + att.reshape(3, hid), atol=1e-12)


def pin_layer_mlp(L):
    """The feed-forward block alone (attention contributes nothing): with gate
    and up reading disjoint halves of the normalised stream, the down projection
    receives silu(gate) * up exactly."""
    import oracle.baton_oracle as O
    rng = np.random.default_rng(4)
    Hq, Hkv, D, hid, F = 2, 2, 8, 16, 8
    gate = np.zeros((F, hid)); gate[:, :8] = np.eye(8)
    up = np.zeros((F, hid)); up[:, 8:] = np.eye(8)
    w = {"norm1": np.ones(hid), "qkv": rng.standard_normal(((Hq + 2 * Hkv) * D, hid)),
         "o": np.zeros((hid, hid)), "norm2": np.ones(hid),
         "gate_up": np.concatenate([gate, up]), "down": np.eye(hid)[:, :F]}
    x = rng.standard_normal((2, hid))
    pb = _batch(O, rng, 1, 2, Hq, Hkv, D, [3, 5])
    out = L.decode_layer(pb, 0, x, w, [3, 5], 10000.0, 0.0)
    h = x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True))
    want = x.copy()
    want[:, :8] += h[:, :8] / (1 + np.exp(-h[:, :8])) * h[:, 8:]
    assert np.allclose(out, want, atol=1e-12)


def pin_layer_stored_bf16(L):
    """decode_layer(stored=bf16) rounds where the GPU stores, worked by hand on
    one query of one cached token (D = hidden = 8, every element alike).
    x = 1.2578125 (bf16 exact), unit gains, eps = 0: the normalised stream is
    exactly 1.  Zero q and k rows make both tokens weigh 1/2; the v rows are
    1.015625 on the diagonal, the cached value 1.0078125, so the attention is
    1.01171875 = 1 + 2^-7 + 2^-8, halfway between two bf16 values: stored, it
    rounds to the even one, 1.015625.  The identity output projection adds it:
    2.2734375, halfway between 2.265625 and 2.28125 (spacing 2^-6 above 2), so
    2.28125.  The zero feed-forward adds nothing.  Unrounded the layer gives
    2.26953125."""
    import oracle.baton_oracle as O
    D = 8
    pb = O.PaddedBatch(1, 1, 1, 1, D, O.BF16)
    pb.embed([0], [1], [np.zeros((1, 1, 1, D), np.uint16)], [np.full((1, 1, 1, D), 0x3F81, np.uint16)])
    qkv = np.zeros((3 * D, D))
    qkv[2 * D:] = np.eye(D) * 1.015625
    w = {"norm1": np.ones(D), "qkv": qkv, "o": np.eye(D), "norm2": np.ones(D),
         "gate_up": np.zeros((2 * D, D)), "down": np.zeros((D, D))}
    x = np.full((1, D), 1.2578125)
    out = L.decode_layer(pb, 0, x, w, [1], 10000.0, 0.0, stored=L.BF16)
    assert np.array_equal(out, np.full((1, D), 2.28125)), out
    pb2 = O.PaddedBatch(1, 1, 1, 1, D, O.BF16)
    pb2.embed([0], [1], [np.zeros((1, 1, 1, D), np.uint16)], [np.full((1, 1, 1, D), 0x3F81, np.uint16)])
    assert np.array_equal(L.decode_layer(pb2, 0, x, w, [1], 10000.0, 0.0), np.full((1, D), 2.26953125))


ALL_PINS = [pin_rmsnorm, pin_rope, pin_silu, pin_linear_and_split, pin_to_bits, pin_layer_residual,
            pin_layer_mlp]
ALL_PINS.append(pin_layer_stored_bf16)
