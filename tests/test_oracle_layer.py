"""The decode-layer oracle against its pins (CPU only), and the pins against
planted mistakes."""
import types

import numpy as np
import pytest

import oracle.llama_layer as L
from tests import oracle_pins_layer as P


@pytest.mark.parametrize("pin", P.ALL_PINS, ids=lambda f: f.__name__)
def test_layer_oracle_pin(pin):
    pin(L)


def _mutant(**overrides):
    m = types.ModuleType("layer_mutant")
    m.__dict__.update(L.__dict__)
    for name, fn in list(L.__dict__.items()):
        if isinstance(fn, types.FunctionType) and fn.__module__ == L.__name__:
            m.__dict__[name] = types.FunctionType(fn.__code__, m.__dict__, name, fn.__defaults__)
    m.__dict__.update(overrides)
    return m


def _rope_interleaved(v, pos, theta):
    v = np.asarray(v, np.float64)
    D = v.shape[-1]
    inv = theta ** (-np.arange(D // 2) * 2.0 / D)
    ang = np.asarray(pos, np.float64)[..., None] * inv
    a, b = v[..., 0::2], v[..., 1::2]
    out = np.empty_like(v)
    out[..., 0::2] = a * np.cos(ang) - b * np.sin(ang)
    out[..., 1::2] = a * np.sin(ang) + b * np.cos(ang)
    return out


def _rope_backwards(v, pos, theta):
    return L.rope(v, -np.asarray(pos, np.float64), theta)


def _rmsnorm_mean(x, g, eps):
    x = np.asarray(x, np.float64)
    return x / (np.abs(np.mean(x, axis=-1, keepdims=True)) + eps + 1e-3) * g


def _silu_sigmoid(z):
    return 1.0 / (1.0 + np.exp(-np.asarray(z, np.float64)))


def _split_kv_swapped(qkv, n_q_heads, n_kv_heads, head_dim):
    q, k, v = L.split_qkv(qkv, n_q_heads, n_kv_heads, head_dim)
    return q, v, k


def _bits_truncate(x, dtype):
    f = np.asarray(x, np.float64).astype(np.float32).view(np.uint32)
    return f.copy() if dtype == L.F32 else (f >> np.uint32(16)).astype(np.uint16)


def _widen_bf16_as_fp16(bits, dtype):
    if dtype == L.BF16:
        return np.asarray(bits).astype(np.uint16).view(np.float16).astype(np.float64)
    return L.widen(bits, dtype)


MUTANTS = {
    "rope pairs interleaved": dict(rope=_rope_interleaved),
    "rope rotates backwards": dict(rope=_rope_backwards),
    "rmsnorm by the mean": dict(rmsnorm=_rmsnorm_mean),
    "silu is a sigmoid": dict(silu=_silu_sigmoid),
    "k and v swapped in the fused projection": dict(split_qkv=_split_kv_swapped),
    "bf16 by truncation": dict(to_bits=_bits_truncate),
    "stored bf16 read back as fp16": dict(widen=_widen_bf16_as_fp16),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_layer_pins_catch_planted_mistake(name):
    M = _mutant(**MUTANTS[name])
    caught = []
    for pin in P.ALL_PINS:
        try:
            pin(M)
        except Exception:
            caught.append(pin.__name__)
    assert caught, f"no pin notices: {name}"
