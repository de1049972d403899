"""Synthetic weights and inputs of a llama2-7b-shaped decoder (the paper's model):
seeded generator values, the same bits on the device and the host.

A weight of input width n is N(0,1) * 2^-k with 2^-k the power of two nearest
1/sqrt(n) (so that activations stay of order one), norm gains are N(0,1); the
scaling is an exact exponent shift of the generator's bf16 values.  Streams:
one per (layer, tensor), one for the decode-step inputs of the residual stream.
"""
import math
from dataclasses import dataclass

import numpy as np

from . import gen

S_WEIGHTS = 64          # + 8 * layer + tensor index
S_X = 11                # residual-stream input of a decode step
TENSORS = ("norm1", "qkv", "o", "norm2", "gate_up", "down")


@dataclass
class ModelShape:
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    theta: float = 10000.0
    eps: float = 1e-5

    def shapes(self):
        hid, F = self.hidden, self.ffn
        return {"norm1": (hid,), "qkv": ((self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim, hid),
                "o": (hid, self.n_q_heads * self.head_dim), "norm2": (hid,), "gate_up": (2 * F, hid),
                "down": (hid, F)}


LLAMA2_7B = ModelShape(4096, 32, 32, 128, 11008)


def scale_exp(shape):
    """k with 2^-k nearest 1/sqrt(input width); 0 for norm gains."""
    return 0 if len(shape) == 1 else round(math.log2(shape[1]) / 2)


def _counter(shape):
    rows, cols = (1, shape[0]) if len(shape) == 1 else shape
    return (1, 1, rows, cols), 0, (0, 0, cols, 1)


def bf16_value(bits):
    """Stored bf16 bits -> float64 (exact)."""
    return (np.asarray(bits).astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def weights_host(seed, m, layer):
    """float64 weights of one layer (exact values of the stored bf16)."""
    out = {}
    for i, name in enumerate(TENSORS):
        shp = m.shapes()[name]
        full, c0, st = _counter(shp)
        bits = gen.fill_host(seed, S_WEIGHTS + 8 * layer + i, "bf16", full, c0, st).reshape(shp)
        out[name] = bf16_value(bits) * 2.0 ** -scale_exp(shp)
    return out


def weights_device(seed, m, layer):
    """bf16 device tensors of one layer."""
    import torch
    out = {}
    for i, name in enumerate(TENSORS):
        shp = m.shapes()[name]
        full, c0, st = _counter(shp)
        t = torch.empty(shp, dtype=torch.bfloat16, device="cuda")
        gen.fill_device(t.data_ptr(), seed, S_WEIGHTS + 8 * layer + i, "bf16", full, c0, st,
                        torch.cuda.current_stream().cuda_stream)
        k = scale_exp(shp)
        if k:
            t.mul_(2.0 ** -k)     # exact: a power of two on bf16 values of order one
        out[name] = t
    return out


def x_counter(step, batch, hidden):
    return step * batch * hidden, (0, 0, hidden, 1)


def x_host(seed, step, batch, hidden):
    c0, st = x_counter(step, batch, hidden)
    return gen.fill_host(seed, S_X, "bf16", (1, 1, batch, hidden), c0, st)[0, 0]


def x_device(seed, step, batch, hidden):
    import torch
    t = torch.empty((batch, hidden), dtype=torch.bfloat16, device="cuda")
    c0, st = x_counter(step, batch, hidden)
    gen.fill_device(t.data_ptr(), seed, S_X, "bf16", (1, 1, batch, hidden), c0, st,
                    torch.cuda.current_stream().cuda_stream)
    return t
