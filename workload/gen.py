"""Seeded, counter-based tensor values for the synthetic decode workloads.

Every tensor element is a pure function of (seed, stream, counter): the value
function lives in csrc/wl_core.h and is compiled for the host (gcc, OpenMP)
and for the GPU (hipcc), so a tensor built on either side has the same bits.
This module holds input generation only; it knows nothing of the re-batching
method.  The pure-Python functions below restate the generator for tiny
known-answer checks of the compiled libraries.
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
HOST_LIB = os.path.join(HERE, "libbaton_wl_host.so")
DEV_LIB = os.path.join(HERE, "libbaton_wl_dev.so")

GAMMA = 0x9E3779B97F4A7C15
M64 = (1 << 64) - 1

# Element codes (csrc/wl_core.h).
F32, BF16 = 0, 1
CODE = {"f32": F32, "bf16": BF16}
STORAGE = {"f32": np.uint32, "bf16": np.uint16}

# Stream ids.
S_LENS = 1        # initial query lengths
S_EVENTS = 2      # evictions, arrivals, inserted lengths
S_PREFILL_K = 3   # keys a prefill instance produced for a query
S_PREFILL_V = 4   # values a prefill instance produced for a query
S_Q = 5           # decode-step queries
S_KNEW = 6        # decode-step keys of the current token
S_VNEW = 7        # decode-step values of the current token
S_QW = 8          # queries of a step that prefills new queries inside the batch
S_KW = 9          # its keys (positions that hold no prompt token)
S_VW = 10         # its values

# Token radix of the prefill counter: prefilled lengths stay below this.
TMAX = 1 << 16


# ---------------------------------------------------------------- reference --
def mix64(z):
    z &= M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def stream_key(seed, stream):
    return mix64(seed * GAMMA + stream)


def draw(key, j):
    return mix64(key + (j + 1) * GAMMA)


def normal_ref(key, c):
    """Pure-Python restatement of wl_normal (returns a Python float, exact)."""
    s = 0
    for j in range(3 * c, 3 * c + 3):
        w = draw(key, j)
        s += sum((w >> sh) & 0xFFFF for sh in (0, 16, 32, 48))
    return (2 * s - 12 * 65535) / 131072.0


def bf16_rne_ref(x):
    u = int(np.array(x, dtype=np.float32).view(np.uint32))
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) & 0xFFFF


# ----------------------------------------------------------------- counters --
def prefill_counter(qid, n_layers, n_kv_heads, head_dim, layer0=0, head0=0, t0=0):
    """(c0, strides) of a query's prefilled K or V laid out [layer][head][t][d]."""
    s2 = head_dim
    s1 = TMAX * head_dim
    s0 = n_kv_heads * s1
    c0 = qid * n_layers * s0 + layer0 * s0 + head0 * s1 + t0 * s2
    return c0, (s0, s1, s2, 1)


def decode_counter(step, layer, n_layers, batch, n_heads, head_dim):
    """(c0, strides) of a decode-step tensor laid out [1][batch][head][d]."""
    c0 = ((step * n_layers + layer) * batch) * n_heads * head_dim
    return c0, (0, n_heads * head_dim, head_dim, 1)


def wide_counter(step, layer, n_layers, batch, n_heads, head_dim):
    """(c0, strides) of a prefill-step tensor laid out [batch][T][head][d] (T < TMAX)."""
    row = n_heads * head_dim
    c0 = ((step * n_layers + layer) * batch) * TMAX * row
    return c0, (TMAX * row, row, head_dim, 1)


def prompt_counter(qid, layer, n_layers, n_kv_heads, head_dim):
    """(c0, strides) of a query's prefilled K or V of one layer laid out [1][t][head][d]:
    the prompt positions of a prefill step carry the values a separate prefill
    of the same query would have produced."""
    c0, (s0, s1, s2, _) = prefill_counter(qid, n_layers, n_kv_heads, head_dim, layer0=layer)
    return c0, (0, s2, s1, 1)


# ------------------------------------------------------------------- host --
_host = None


def host_lib():
    global _host
    if _host is None:
        if not os.path.exists(HOST_LIB):
            raise RuntimeError(f"{HOST_LIB} is missing: run workload/build.py")
        lib = ctypes.CDLL(HOST_LIB)
        u64, i64 = ctypes.c_uint64, ctypes.c_int64
        lib.wl_host_fill.restype = ctypes.c_int
        lib.wl_host_fill.argtypes = [u64, ctypes.c_int, ctypes.c_void_p, i64, i64, i64, i64,
                                     u64, u64, u64, u64, u64]
        lib.wl_host_stream_key.restype = u64
        lib.wl_host_stream_key.argtypes = [u64, u64]
        lib.wl_host_draw.restype = u64
        lib.wl_host_draw.argtypes = [u64, u64]
        lib.wl_host_normal.restype = ctypes.c_float
        lib.wl_host_normal.argtypes = [u64, u64]
        lib.wl_host_bf16_rne.restype = ctypes.c_uint16
        lib.wl_host_bf16_rne.argtypes = [ctypes.c_float]
        _host = lib
    return _host


def fill_host(seed, stream, dtype, shape, c0, strides):
    """Host array of stored bits (uint32 for f32, uint16 for bf16) of the given 4-D shape."""
    shape = tuple(int(n) for n in shape)
    assert len(shape) == 4 and len(strides) == 4
    out = np.empty(shape, dtype=STORAGE[dtype])
    key = stream_key(seed, stream)
    rc = host_lib().wl_host_fill(key, CODE[dtype], out.ctypes.data, *shape,
                                 c0 & M64, *(s & M64 for s in strides))
    if rc != 0:
        raise RuntimeError(f"wl_host_fill failed ({rc})")
    return out


def prefill_host(seed, which, qid, n_layers, n_kv_heads, length, head_dim, dtype):
    """A query's prefilled K (which='k') or V (which='v'): bits [layer][head][length][d]."""
    stream = S_PREFILL_K if which == "k" else S_PREFILL_V
    c0, st = prefill_counter(qid, n_layers, n_kv_heads, head_dim)
    return fill_host(seed, stream, dtype, (n_layers, n_kv_heads, length, head_dim), c0, st)


def decode_host(seed, stream, step, layer, n_layers, batch, n_heads, head_dim, dtype):
    """Decode-step tensor (q, k_new or v_new): bits [batch][head][d]."""
    c0, st = decode_counter(step, layer, n_layers, batch, n_heads, head_dim)
    return fill_host(seed, stream, dtype, (1, batch, n_heads, head_dim), c0, st)[0]


def prefill_step_host(seed, which, step, layer, n_layers, batch, T, n_heads, head_dim, dtype,
                      inserted=()):
    """Inputs of a step that prefills queries inside the batch: which in 'q', 'k',
    'v'; bits [batch][T][head][d].  inserted: (slot, qid, prompt length) of the
    queries prefilled in it; their prompt positions' keys and values are their
    prefilled ones."""
    stream = {"q": S_QW, "k": S_KW, "v": S_VW}[which]
    c0, st = wide_counter(step, layer, n_layers, batch, n_heads, head_dim)
    out = fill_host(seed, stream, dtype, (batch, T, n_heads, head_dim), c0, st)
    if which != "q":
        ps = S_PREFILL_K if which == "k" else S_PREFILL_V
        for slot, qid, n in inserted:
            c0, st = prompt_counter(qid, layer, n_layers, n_heads, head_dim)
            out[slot, T - n:] = fill_host(seed, ps, dtype, (1, n, n_heads, head_dim), c0, st)[0]
    return out


# ----------------------------------------------------------------- device --
_dev = None


def dev_lib():
    global _dev
    if _dev is None:
        if not os.path.exists(DEV_LIB):
            raise RuntimeError(f"{DEV_LIB} is missing: run workload/build.py")
        lib = ctypes.CDLL(DEV_LIB)
        u64, i64 = ctypes.c_uint64, ctypes.c_int64
        lib.wl_device_read_stream.restype = ctypes.c_int
        lib.wl_device_read_stream.argtypes = [ctypes.c_void_p, i64, ctypes.c_void_p, ctypes.c_void_p]
        lib.wl_device_fill.restype = ctypes.c_int
        lib.wl_device_fill.argtypes = [u64, ctypes.c_int, ctypes.c_void_p, i64, i64, i64, i64,
                                       u64, u64, u64, u64, u64, ctypes.c_void_p]
        _dev = lib
    return _dev


def fill_device(ptr, seed, stream, dtype, shape, c0, strides, hip_stream=0):
    """Device twin of fill_host, written into device memory at `ptr` on `hip_stream`."""
    shape = tuple(int(n) for n in shape)
    key = stream_key(seed, stream)
    rc = dev_lib().wl_device_fill(key, CODE[dtype], ctypes.c_void_p(ptr), *shape, c0 & M64,
                                  *(s & M64 for s in strides), ctypes.c_void_p(hip_stream))
    if rc != 0:
        raise RuntimeError(f"wl_device_fill failed ({rc})")
