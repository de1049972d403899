"""CPU oracle of a whole decode layer around the re-batched attention -- TEST
INFRASTRUCTURE ONLY (tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg; the library never imports it and shares no code with it).

The paper serves llama2-7b-chat-hf (sec. 5, experimental setup) and describes
its layers in general terms (sec. 2.1, "General architecture"): the input is
linearly transformed by W^Q, W^K, W^V into queries, keys and values, the
attention output is their scaled-dot-product softmax average, and
feed-forward networks sit between attention blocks.  The layer below is that
model's decoder layer, written from the definitions of its parts:

* RMS normalisation before each block: y = x / sqrt(mean(x^2) + eps) * g;
* rotary position embedding of queries and keys, in the rotate-half pairing of
  the Hugging Face checkpoint (dimension i pairs with i + D/2), angle
  pos * theta^(-2i/D) for pair i;
* attention over each query's own tokens (baton_oracle.attend, through the
  PaddedBatch so that the cache evolves as the method says);
* output projection added to the residual stream;
* gated feed-forward: down( silu(gate(h)) * up(h) ), silu(z) = z / (1 + e^-z),
  added to the residual stream.

Every function takes and returns float64 arrays; linear layers compute
x @ W^T with W stored [out][in], as the checkpoint stores them.  Readings
where the paper is silent: the position of a decode token is the number of
tokens its query already has (the token count of the slot, holes excluded);
each GPU operation rounds its output to bf16, so the parity tests compare
every operation on the GPU's own inputs, and the whole layer with a
tolerance for the accumulated roundings.
"""
import numpy as np

from .baton_oracle import BF16, F32, widen


def rmsnorm(x, g, eps):
    """Rows of x normalised by their root mean square, scaled by g."""
    x = np.asarray(x, np.float64)
    rms = np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return x / rms * np.asarray(g, np.float64)


def rope(v, pos, theta):
    """Rotary embedding of v [..., D] at position pos (scalar or broadcastable
    to v[..., 0]); pair (i, i + D/2) rotated by pos * theta^(-2i/D)."""
    v = np.asarray(v, np.float64)
    D = v.shape[-1]
    half = D // 2
    inv = theta ** (-np.arange(half, dtype=np.float64) * 2.0 / D)
    ang = np.asarray(pos, np.float64)[..., None] * inv
    c, s = np.cos(ang), np.sin(ang)
    a, b = v[..., :half], v[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def silu(z):
    z = np.asarray(z, np.float64)
    return z / (1.0 + np.exp(-z))


def linear(x, w):
    """x [..., in] times the stored weight [out][in], transposed."""
    return np.asarray(x, np.float64) @ np.asarray(w, np.float64).T


def split_qkv(qkv, n_q_heads, n_kv_heads, head_dim):
    """The fused projection's output [B][(Hq + 2 Hkv) * D] as q [B][Hq][D],
    k [B][Hkv][D], v [B][Hkv][D] (q rows first, then k, then v)."""
    B = qkv.shape[0]
    q = qkv[:, :n_q_heads * head_dim].reshape(B, n_q_heads, head_dim)
    k = qkv[:, n_q_heads * head_dim:(n_q_heads + n_kv_heads) * head_dim].reshape(B, n_kv_heads, head_dim)
    v = qkv[:, (n_q_heads + n_kv_heads) * head_dim:].reshape(B, n_kv_heads, head_dim)
    return q, k, v


def to_bits(x, dtype):
    """float64 -> stored bits, rounding to nearest even (as the GPU stores)."""
    f = np.asarray(x, np.float64).astype(np.float32)
    u = f.view(np.uint32)
    if dtype == F32:
        return u.copy()
    return ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)


def decode_layer(pb, layer, x, w, positions, theta, eps, scale=None, stored=None):
    """One decode layer of the batch in float64.

    pb: the baton_oracle.PaddedBatch (its decode_layer appends this layer's
    keys/values); x [B][hidden] float64 (free rows ignored); w: dict of float64
    weights: norm1 [hidden], qkv [(Hq + 2 Hkv) D][hidden], o [hidden][Hq D],
    norm2 [hidden], gate_up [2 F][hidden] (gate rows first), down [hidden][F];
    positions [B]: each slot's token count.  Keys and values enter the cache
    rounded to the cache's element type, as the GPU stores them.  Returns the
    new residual stream [B][hidden] (free rows unchanged).

    stored: None, or an element type in which every intermediate is stored
    between operations (the GPU's bf16 activations); the rounding then happens
    where the GPU rounds, and only the order of accumulation differs."""
    Hq, Hkv, D = pb.Hq, pb.Hkv, pb.D
    r = (lambda v: v) if stored is None else (lambda v: widen(to_bits(v, stored), stored))
    h = r(rmsnorm(x, w["norm1"], eps))
    q, k, v = split_qkv(r(linear(h, w["qkv"])), Hq, Hkv, D)
    pos = np.asarray(positions, np.float64)[:, None]
    q, k = rope(q, pos, theta), rope(k, pos, theta)
    att = r(pb.decode_layer(layer, to_bits(q, pb.dtype), to_bits(k, pb.dtype), to_bits(v, pb.dtype), scale))
    x = r(x + linear(att.reshape(att.shape[0], Hq * D), w["o"]))
    h2 = r(rmsnorm(x, w["norm2"], eps))
    gu = r(linear(h2, w["gate_up"]))
    F = gu.shape[-1] // 2
    return r(x + linear(r(silu(gu[:, :F]) * gu[:, F:]), w["down"]))
