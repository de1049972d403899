"""Python binding of libbaton.so: the C ABI of include/baton.h, same names.

Argument marshalling only -- every step of the re-batched decode runs in the
library's HIP kernels.  Device buffers may be passed as integers (device
addresses) or as objects with a data_ptr() method (torch tensors); streams as
integers (hipStream_t) or objects with a cuda_stream attribute.  A non-OK
status raises BatonError.  The library must have been built
(paper_2410_18701_amd/build.py); there is no fallback.
"""
import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libbaton.so")

BATON_OK, BATON_EINVAL, BATON_ESLOT, BATON_ECAPACITY, BATON_EDTYPE, BATON_ESTATE, BATON_EHIP, \
    BATON_ESCRATCH = range(8)
STATUS_NAMES = ["BATON_OK", "BATON_EINVAL", "BATON_ESLOT", "BATON_ECAPACITY", "BATON_EDTYPE",
                "BATON_ESTATE", "BATON_EHIP", "BATON_ESCRATCH"]
BATON_SCRATCH_BYTES = 64 << 20
BATON_GEMM_MAX_ROWS = 256
BATON_F32, BATON_BF16 = 0, 1
BATON_FILL_NEG_INF_F32 = 0xFF800000
BATON_FILL_NEG_INF_BF16 = 0xFF80
BATON_MAX_BATCH = 512
BATON_MAX_PREFILL = 64
BATON_MAX_HOLES = 64
BATON_CREATE_ASSUME_FILLED = 1
BATON_RELEASE = 1
BATON_SCRUB = 2


class baton_cache_desc(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("n_layers", ctypes.c_int32), ("batch", ctypes.c_int32),
                ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("capacity", ctypes.c_int64),
                ("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("fill_bits", ctypes.c_uint32),
                ("layer_stride", ctypes.c_int64)]


class BatonError(RuntimeError):
    def __init__(self, status, call):
        self.status = status
        name = STATUS_NAMES[status] if 0 <= status < len(STATUS_NAMES) else str(status)
        super().__init__(f"{call}: {name} ({baton_status_string(status)})")


_lib = None


def lib():
    """The loaded libbaton.so; raises if it was not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2410_18701_amd/build.py "
                               "(there is no fallback path)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, u32, st = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_int
        P = ctypes.POINTER
        L.baton_cache_create.argtypes = [P(baton_cache_desc), u32, vp, P(vp)]
        L.baton_cache_destroy.argtypes = [vp]
        L.baton_kv_evict.argtypes = [vp, P(i32), i32, u32, vp]
        L.baton_kv_embed.argtypes = [vp, P(i32), i32, P(i32), P(vp), P(vp), vp]
        L.baton_kv_extract.argtypes = [vp, P(i32), i32, P(vp), P(vp), vp]
        L.baton_shape_insert.argtypes = [vp, P(i32), i32, P(i32)]
        L.baton_kv_move.argtypes = [vp, P(i32), P(i32), i32, vp]
        L.baton_cache_tokens.argtypes = [vp, P(i32)]
        L.baton_build_mask.argtypes = [vp, vp, i64, vp]
        L.baton_decode_attn_workspace_bytes.argtypes = [vp]
        L.baton_decode_attn_workspace_bytes.restype = ctypes.c_size_t
        L.baton_decode_attn.argtypes = [vp, i32, vp, vp, vp, vp, ctypes.c_float, vp, ctypes.c_size_t, vp]
        L.baton_decode_attn_noalloc.argtypes = [vp, i32, vp, vp, vp, vp, ctypes.c_float, vp]
        L.baton_step_advance.argtypes = [vp]
        L.baton_cache_flush.argtypes = [vp, vp]
        L.baton_cache_query.argtypes = [vp, P(i64), P(i64), P(i32)]
        L.baton_set_split_tokens.argtypes = [vp, i32]
        L.baton_linear_packed_bytes.argtypes = [i32, i32]
        L.baton_linear_packed_bytes.restype = ctypes.c_size_t
        L.baton_linear_pack.argtypes = [i32, vp, vp, i32, i32, vp]
        L.baton_linear_packed.argtypes = [i32, vp, vp, vp, i32, i32, i32, i32, vp, ctypes.c_size_t, vp]
        L.baton_linear_packed_rmsnorm.argtypes = [i32, vp, vp, vp, i32, i32, i32, i32, vp, ctypes.c_float, vp,
                                                  vp, ctypes.c_size_t, vp]
        L.baton_linear_packed_silu.argtypes = [i32, vp, vp, vp, i32, i32, i32, vp]
        L.baton_rmsnorm.argtypes = [i32, vp, vp, vp, i32, i32, ctypes.c_float, vp]
        L.baton_rope_qkv.argtypes = [vp, vp, vp, vp, vp, ctypes.c_float, vp]
        L.baton_silu_mul.argtypes = [i32, vp, vp, i32, i32, vp]
        L.baton_status_string.argtypes = [st]
        L.baton_status_string.restype = ctypes.c_char_p
        for name in ("baton_cache_create", "baton_cache_destroy", "baton_kv_evict", "baton_kv_embed",
                     "baton_kv_extract",
                     "baton_build_mask", "baton_decode_attn", "baton_decode_attn_noalloc", "baton_step_advance",
                     "baton_cache_query", "baton_set_split_tokens", "baton_cache_flush",
                     "baton_shape_insert", "baton_cache_tokens", "baton_kv_move", "baton_linear_pack", "baton_linear_packed",
                     "baton_linear_packed_rmsnorm", "baton_linear_packed_silu",
                     "baton_rmsnorm", "baton_rope_qkv", "baton_silu_mul"):
            getattr(L, name).restype = st
        _lib = L
    return _lib


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(s):
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _check(status, call):
    if status != BATON_OK:
        raise BatonError(status, call)


def _i32s(values):
    values = [int(v) for v in values]
    return (ctypes.c_int32 * max(1, len(values)))(*values), len(values)


def baton_status_string(status):
    return lib().baton_status_string(int(status)).decode()


def baton_cache_create(desc, flags=0, stream=None):
    """Returns the handle (an opaque integer)."""
    out = ctypes.c_void_p()
    _check(lib().baton_cache_create(ctypes.byref(desc), flags, _stream(stream), ctypes.byref(out)),
           "baton_cache_create")
    return out.value


def baton_cache_destroy(cache):
    _check(lib().baton_cache_destroy(cache), "baton_cache_destroy")


def baton_kv_evict(cache, slots, flags=BATON_RELEASE | BATON_SCRUB, stream=None):
    arr, n = _i32s(slots)
    _check(lib().baton_kv_evict(cache, arr, n, flags, _stream(stream)), "baton_kv_evict")


def baton_kv_embed(cache, slots, lens, k_src, v_src, stream=None):
    s_arr, n = _i32s(slots)
    l_arr, nl = _i32s(lens)
    if nl != n or len(k_src) != n or len(v_src) != n:
        raise ValueError("slots, lens, k_src and v_src must have the same length")
    ks = (ctypes.c_void_p * max(1, n))(*[_ptr(x) for x in k_src])
    vs = (ctypes.c_void_p * max(1, n))(*[_ptr(x) for x in v_src])
    _check(lib().baton_kv_embed(cache, s_arr, n, l_arr, ks, vs, _stream(stream)), "baton_kv_embed")


def baton_kv_extract(cache, slots, k_dst, v_dst, stream=None):
    s_arr, n = _i32s(slots)
    if len(k_dst) != n or len(v_dst) != n:
        raise ValueError("slots, k_dst and v_dst must have the same length")
    ks = (ctypes.c_void_p * max(1, n))(*[_ptr(x) for x in k_dst])
    vs = (ctypes.c_void_p * max(1, n))(*[_ptr(x) for x in v_dst])
    _check(lib().baton_kv_extract(cache, s_arr, n, ks, vs, _stream(stream)), "baton_kv_extract")


def baton_kv_move(cache, src, dst, stream=None):
    s_arr, n = _i32s(src)
    d_arr, nd = _i32s(dst)
    if nd != n:
        raise ValueError("src and dst must have the same length")
    _check(lib().baton_kv_move(cache, s_arr, d_arr, n, _stream(stream)), "baton_kv_move")


def baton_shape_insert(cache, slots, lens):
    s_arr, n = _i32s(slots)
    l_arr, nl = _i32s(lens)
    if nl != n:
        raise ValueError("slots and lens must have the same length")
    _check(lib().baton_shape_insert(cache, s_arr, n, l_arr), "baton_shape_insert")


def baton_cache_tokens(cache, batch):
    """Per-slot token counts (list)."""
    out = (ctypes.c_int32 * batch)()
    _check(lib().baton_cache_tokens(cache, out), "baton_cache_tokens")
    return list(out)


def baton_build_mask(cache, mask, ld, stream=None):
    _check(lib().baton_build_mask(cache, _ptr(mask), ld, _stream(stream)), "baton_build_mask")


def baton_decode_attn_workspace_bytes(cache):
    return lib().baton_decode_attn_workspace_bytes(cache)


def baton_decode_attn(cache, layer, q, k_new, v_new, out, scale, ws, ws_bytes, stream=None):
    _check(lib().baton_decode_attn(cache, layer, _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(out),
                                   float(scale), _ptr(ws), ws_bytes, _stream(stream)),
           "baton_decode_attn")


def baton_decode_attn_noalloc(cache, layer, q, k_new, v_new, out, scale, stream=None):
    _check(lib().baton_decode_attn_noalloc(cache, layer, _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(out),
                                           float(scale), _stream(stream)),
           "baton_decode_attn_noalloc")


def baton_cache_flush(cache, stream=None):
    _check(lib().baton_cache_flush(cache, _stream(stream)), "baton_cache_flush")


def baton_step_advance(cache):
    _check(lib().baton_step_advance(cache), "baton_step_advance")


def baton_cache_query(cache, batch):
    """Returns (L, base, lens list)."""
    L = ctypes.c_int64()
    base = ctypes.c_int64()
    lens = (ctypes.c_int32 * batch)()
    _check(lib().baton_cache_query(cache, ctypes.byref(L), ctypes.byref(base), lens),
           "baton_cache_query")
    return L.value, base.value, list(lens)


def baton_set_split_tokens(cache, tokens):
    _check(lib().baton_set_split_tokens(cache, tokens), "baton_set_split_tokens")


# ---- decode layer around the attention ----
def baton_linear_packed_bytes(out_dim, in_dim):
    return lib().baton_linear_packed_bytes(out_dim, in_dim)


def baton_linear_pack(dtype, w, wp, out_dim, in_dim, stream=None):
    _check(lib().baton_linear_pack(dtype, _ptr(w), _ptr(wp), out_dim, in_dim, _stream(stream)), "baton_linear_pack")


def baton_linear_packed(dtype, x, wp, y, rows, out_dim, in_dim, accumulate, ws, ws_bytes, stream=None):
    _check(lib().baton_linear_packed(dtype, _ptr(x), _ptr(wp), _ptr(y), rows, out_dim, in_dim, int(accumulate),
                                     _ptr(ws), ws_bytes, _stream(stream)), "baton_linear_packed")


def baton_linear_packed_rmsnorm(dtype, x, wp, y, rows, out_dim, in_dim, accumulate, gain, eps, y_norm, ws,
                                ws_bytes, stream=None):
    _check(lib().baton_linear_packed_rmsnorm(dtype, _ptr(x), _ptr(wp), _ptr(y), rows, out_dim, in_dim,
                                             int(accumulate), _ptr(gain), float(eps), _ptr(y_norm), _ptr(ws),
                                             ws_bytes, _stream(stream)), "baton_linear_packed_rmsnorm")


def baton_linear_packed_silu(dtype, x, wp, y, rows, out_dim, in_dim, stream=None):
    _check(lib().baton_linear_packed_silu(dtype, _ptr(x), _ptr(wp), _ptr(y), rows, out_dim, in_dim,
                                          _stream(stream)), "baton_linear_packed_silu")


def baton_rmsnorm(dtype, x, gain, y, rows, dim, eps, stream=None):
    _check(lib().baton_rmsnorm(dtype, _ptr(x), _ptr(gain), _ptr(y), rows, dim, float(eps), _stream(stream)),
           "baton_rmsnorm")


def baton_rope_qkv(cache, qkv, q, k_new, v_new, theta, stream=None):
    _check(lib().baton_rope_qkv(cache, _ptr(qkv), _ptr(q), _ptr(k_new), _ptr(v_new), float(theta),
                                _stream(stream)), "baton_rope_qkv")


def baton_silu_mul(dtype, gate_up, out, rows, dim, stream=None):
    _check(lib().baton_silu_mul(dtype, _ptr(gate_up), _ptr(out), rows, dim, _stream(stream)), "baton_silu_mul")
