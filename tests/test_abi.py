"""The C ABI on the CPU: the library loads, exports every symbol of
include/baton.h, and its host-side checks refuse bad calls before any device
work (no GPU is touched: every call here returns before enqueueing)."""
import ctypes
import os
import re

import pytest

from paper_2410_18701_amd import baton as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "baton.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(baton_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert "baton_decode_attn" in names and "baton_kv_embed" in names
    lib = B.lib()
    for n in names:
        assert hasattr(lib, n), f"{n} declared in baton.h but not exported"


def test_status_strings():
    for s in range(8):
        assert B.baton_status_string(s) != "unknown status"
    assert B.baton_status_string(99) == "unknown status"


FAKE_K, FAKE_V = 0x10000, 0x10000000   # never dereferenced: every call below fails host checks


def desc(**kw):
    d = dict(dtype=B.BATON_BF16, n_layers=2, batch=4, n_q_heads=8, n_kv_heads=2, head_dim=128,
             capacity=300, k=FAKE_K, v=FAKE_V, fill_bits=B.BATON_FILL_NEG_INF_BF16)
    d.update(kw)
    return B.baton_cache_desc(**d)


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=7), B.BATON_EDTYPE), (dict(head_dim=96), B.BATON_EDTYPE),
    (dict(n_q_heads=6, n_kv_heads=4), B.BATON_EDTYPE), (dict(n_q_heads=32, n_kv_heads=2), B.BATON_EDTYPE),
    (dict(batch=0), B.BATON_EINVAL), (dict(batch=513), B.BATON_EINVAL), (dict(capacity=1), B.BATON_EINVAL),
    (dict(n_layers=0), B.BATON_EINVAL), (dict(k=0), B.BATON_EINVAL), (dict(v=FAKE_V + 8), B.BATON_EINVAL),
    # one layer's rows are 4 x 2 x 300 x 128 elements (307,200 = 614,400 bytes)
    (dict(layer_stride=307200 - 8), B.BATON_EINVAL),                   # below one layer
    (dict(layer_stride=307200 + 4), B.BATON_EINVAL),                   # 8 bytes: not whole vectors
    (dict(v=FAKE_K + 16), B.BATON_EINVAL),                             # overlaps k
    (dict(v=FAKE_K + 614400, layer_stride=2 * 307200 - 8), B.BATON_EINVAL),   # interleaved, overlapping
    (dict(layer_stride=-307200), B.BATON_EINVAL),                      # negative
    (dict(layer_stride=1 << 60), B.BATON_EINVAL),                      # spans beyond any memory
    (dict(n_kv_heads=1 << 30, n_q_heads=1 << 30), B.BATON_EINVAL),     # rows beyond any memory
])
def test_create_rejects(kw, status):
    with pytest.raises(B.BatonError) as e:
        B.baton_cache_create(desc(**kw), B.BATON_CREATE_ASSUME_FILLED)
    assert e.value.status == status


@pytest.mark.parametrize("kw", [
    dict(v=FAKE_K + 614400, layer_stride=2 * 307200),        # [n_layers][2][...]: v after k's layer
    dict(v=FAKE_K + 614400 * 4, layer_stride=2 * 307200),    # v after the whole of k
    dict(v=FAKE_K + 2 * 614400),                               # packed, v right after k
    dict(layer_stride=307200),                                 # packed, stride given
])
def test_create_accepts_layouts(kw):
    B.baton_cache_destroy(B.baton_cache_create(desc(**kw), B.BATON_CREATE_ASSUME_FILLED))


def test_host_checks_leave_state_unchanged():
    h = B.baton_cache_create(desc(), B.BATON_CREATE_ASSUME_FILLED)
    try:
        assert B.baton_cache_query(h, 4) == (0, 0, [0, 0, 0, 0])
        assert B.baton_decode_attn_workspace_bytes(h) > 0

        def status(fn, *a):
            with pytest.raises(B.BatonError) as e:
                fn(*a)
            return e.value.status

        assert status(B.baton_kv_evict, h, [1]) == B.BATON_ESLOT          # free slot
        assert status(B.baton_kv_evict, h, [4]) == B.BATON_EINVAL         # out of range
        assert status(B.baton_kv_evict, h, [0, 0]) == B.BATON_EINVAL      # duplicate
        assert status(B.baton_kv_evict, h, [], 4) == B.BATON_EINVAL       # unknown flag
        assert status(B.baton_kv_evict, h, [1], B.BATON_SCRUB) == B.BATON_ESLOT
        B.baton_kv_evict(h, [], B.BATON_RELEASE | B.BATON_SCRUB)          # both flags, no slot
        B.baton_kv_evict(h, [], 0)                                         # neither
        assert status(B.baton_kv_embed, h, [0], [0], [FAKE_K], [FAKE_V]) == B.BATON_EINVAL   # empty query
        assert status(B.baton_kv_embed, h, [0], [300], [FAKE_K], [FAKE_V]) == B.BATON_ECAPACITY  # 300+1 > 300
        assert status(B.baton_kv_embed, h, [0, 0], [3, 3], [FAKE_K] * 2, [FAKE_V] * 2) == B.BATON_EINVAL
        assert status(B.baton_kv_embed, h, [0], [3], [0], [FAKE_V]) == B.BATON_EINVAL      # null source
        assert status(B.baton_kv_embed, h, [0], [3], [FAKE_K + 4], [FAKE_V]) == B.BATON_EINVAL  # misaligned
        assert status(B.baton_kv_extract, h, [0], [FAKE_K], [FAKE_V]) == B.BATON_ESLOT   # free slot
        assert status(B.baton_kv_extract, h, [0, 0], [FAKE_K] * 2, [FAKE_V] * 2) == B.BATON_EINVAL
        assert status(B.baton_kv_extract, h, [0], [FAKE_K + 8], [FAKE_V]) == B.BATON_EINVAL
        B.baton_kv_extract(h, [], [], [])                                  # nothing to do
        B.baton_cache_flush(h)                                             # nothing owed
        assert status(B.baton_step_advance, h) == B.BATON_ESTATE          # no layer decoded
        ws = B.baton_decode_attn_workspace_bytes(h)
        assert status(B.baton_decode_attn, h, 2, FAKE_K, FAKE_K, FAKE_K, FAKE_K, 0.0, FAKE_V, ws) == B.BATON_EINVAL
        assert status(B.baton_decode_attn, h, 0, 0, FAKE_K, FAKE_K, FAKE_K, 0.0, FAKE_V, ws) == B.BATON_EINVAL
        assert status(B.baton_decode_attn, h, 0, FAKE_K, FAKE_K, FAKE_K, FAKE_K, 0.0, FAKE_V, ws - 1) == B.BATON_EINVAL
        assert status(B.baton_decode_attn, h, 0, FAKE_K, FAKE_K, FAKE_K, FAKE_K, float("nan"), FAKE_V, ws) == B.BATON_EINVAL
        nd = B.baton_decode_attn_noalloc
        assert status(nd, h, 2, FAKE_K, FAKE_K, FAKE_K, FAKE_K, 0.0) == B.BATON_EINVAL          # layer
        assert status(nd, h, 0, FAKE_K, 0, FAKE_K, FAKE_K, 0.0) == B.BATON_EINVAL               # null k_new
        assert status(nd, h, 0, FAKE_K, FAKE_K, FAKE_K, FAKE_K + 2, 0.0) == B.BATON_EINVAL      # misaligned
        assert status(nd, h, 0, FAKE_K, FAKE_K, FAKE_K, FAKE_K, float("inf"), 0) == B.BATON_EINVAL
        assert status(B.baton_build_mask, h, 0, 1) == B.BATON_EINVAL
        assert status(B.baton_build_mask, h, FAKE_K, 0) == B.BATON_EINVAL   # ld < L + 1
        assert status(B.baton_set_split_tokens, h, 100) == B.BATON_EINVAL
        assert B.baton_cache_query(h, 4) == (0, 0, [0, 0, 0, 0])
        assert status(B.baton_kv_move, h, [1], [2]) == B.BATON_ESLOT              # source free
        assert status(B.baton_kv_move, h, [1], [1]) == B.BATON_EINVAL             # listed twice
        assert status(B.baton_kv_move, h, [0], [7]) == B.BATON_EINVAL             # out of range
        B.baton_kv_move(h, [], [])                                                 # nothing to do
        # in-batch prefill registration (host metadata only)
        assert status(B.baton_shape_insert, h, [], []) == B.BATON_EINVAL          # nothing to insert
        assert status(B.baton_shape_insert, h, [1, 1], [3, 3]) == B.BATON_EINVAL  # duplicate
        assert status(B.baton_shape_insert, h, [1], [0]) == B.BATON_EINVAL        # empty prompt
        assert status(B.baton_shape_insert, h, [5], [3]) == B.BATON_EINVAL        # out of range
        assert status(B.baton_shape_insert, h, [1], [301]) == B.BATON_ECAPACITY   # L + T > capacity
        assert status(B.baton_shape_insert, h, list(range(4)) * 17, [1] * 68) == B.BATON_EINVAL  # > max
        B.baton_shape_insert(h, [1, 3], [7, 300])
        assert status(B.baton_kv_evict, h, []) == B.BATON_ESTATE                   # prefill registered
        assert status(B.baton_kv_embed, h, [], [], [], []) == B.BATON_ESTATE
        assert status(B.baton_build_mask, h, FAKE_K, 299) == B.BATON_EINVAL       # ld < L + T
        assert B.baton_cache_tokens(h, 4) == [0, 0, 0, 0]
        B.baton_shape_insert(h, [2], [1])                                          # replaces it
        assert status(B.baton_kv_evict, h, []) == B.BATON_ESTATE
        B.baton_set_split_tokens(h, 64)
        assert B.baton_decode_attn_workspace_bytes(h) > ws                # more, smaller splits
    finally:
        B.baton_cache_destroy(h)


def test_packed_linear_host_checks():
    """Sizes of the packed weight, and the checks of baton_linear_pack /
    baton_linear_packed (fake aligned addresses: every call fails before any
    device work)."""
    assert B.baton_linear_packed_bytes(4096, 4096) == 4096 * 4096 * 2
    assert B.baton_linear_packed_bytes(1000, 1000) == 1008 * 1024 * 2   # 16-row slices, 32-column blocks
    assert B.baton_linear_packed_bytes(0, 64) == 0
    X, W, Y = 0x10000, 0x20000, 0x30000

    def status(f, *a):
        try:
            f(*a)
        except B.BatonError as e:
            return e.status
        return B.BATON_OK

    assert status(B.baton_linear_pack, B.BATON_BF16, 0, W, 64, 64) == B.BATON_EINVAL            # null
    assert status(B.baton_linear_pack, B.BATON_BF16, X + 8, W, 64, 64) == B.BATON_EINVAL        # misaligned
    assert status(B.baton_linear_pack, B.BATON_BF16, X, W, 64, 60) == B.BATON_EINVAL            # in % 8
    assert status(B.baton_linear_pack, B.BATON_F32, X, W, 64, 64) == B.BATON_EDTYPE
    lp = B.baton_linear_packed
    assert status(lp, B.BATON_BF16, X, W, Y, 257, 64, 64, 0, 0, 0) == B.BATON_EINVAL          # rows > 256
    assert status(lp, B.BATON_BF16, X, W, Y, 0, 64, 64, 0, 0, 0) == B.BATON_EINVAL            # rows < 1
    assert status(lp, B.BATON_BF16, X, W, 0, 8, 64, 64, 0, 0, 0) == B.BATON_EINVAL            # null y
    assert status(lp, B.BATON_BF16, X, W + 4, Y, 8, 64, 64, 0, 0, 0) == B.BATON_EINVAL        # misaligned
    assert status(lp, B.BATON_BF16, X, W, Y, 8, 68, 64, 0, 0, 0) == B.BATON_EINVAL            # out % 8
    assert status(lp, B.BATON_BF16, X, W, Y, 8, 64, 64, 2, 0, 0) == B.BATON_EINVAL            # accumulate
    assert status(lp, B.BATON_BF16, X, W, Y, 8, 64, 64, 0, 0, 1024) == B.BATON_EINVAL         # ws_bytes, no ws
    assert status(lp, B.BATON_F32, X, W, Y, 8, 64, 64, 0, 0, 0) == B.BATON_EDTYPE
    G, N = 0x40000, 0x50000
    lpn = B.baton_linear_packed_rmsnorm
    assert status(lpn, B.BATON_BF16, X, W, Y, 8, 64, 64, 1, 0, 1e-5, N, 0, 0) == B.BATON_EINVAL      # null gain
    assert status(lpn, B.BATON_BF16, X, W, Y, 8, 64, 64, 1, G, 1e-5, 0, 0, 0) == B.BATON_EINVAL      # null y_norm
    assert status(lpn, B.BATON_BF16, X, W, Y, 8, 64, 64, 1, G + 8, 1e-5, N, 0, 0) == B.BATON_EINVAL  # misaligned
    assert status(lpn, B.BATON_BF16, X, W, Y, 8, 64, 64, 1, G, -1.0, N, 0, 0) == B.BATON_EINVAL      # eps < 0
    assert status(lpn, B.BATON_BF16, X, W, Y, 257, 64, 64, 1, G, 1e-5, N, 0, 0) == B.BATON_EINVAL    # rows > 256
    assert status(lpn, B.BATON_F32, X, W, Y, 8, 64, 64, 1, G, 1e-5, N, 0, 0) == B.BATON_EDTYPE
    lps = B.baton_linear_packed_silu
    assert status(lps, B.BATON_BF16, X, W, 0, 8, 64, 64) == B.BATON_EINVAL       # null y
    assert status(lps, B.BATON_BF16, X, W, Y, 8, 48, 64) == B.BATON_EINVAL       # out % 32
    assert status(lps, B.BATON_BF16, X, W, Y, 257, 64, 64) == B.BATON_EINVAL     # rows > 256
    assert status(lps, B.BATON_BF16, X, W + 8, Y, 8, 64, 64) == B.BATON_EINVAL   # misaligned
    assert status(lps, B.BATON_BF16, X, W, Y, 8, 64, 60) == B.BATON_EINVAL       # in % 8
    assert status(lps, B.BATON_F32, X, W, Y, 8, 64, 64) == B.BATON_EDTYPE
