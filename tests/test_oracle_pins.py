"""The oracle against its pins (CPU only), and the pins against planted mistakes."""
import copy
import types

import numpy as np
import pytest

import oracle.baton_oracle as O
from tests import oracle_pins as P


@pytest.mark.parametrize("pin", P.ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(pin):
    pin(O)


# ------------------------------------------------------------ mutations --
# Each mutant is the oracle with one plausible mistake; some pin must fail on it.

def _mutant(**overrides):
    """A copy of the oracle module whose functions and methods resolve names in the
    copy, so that one overridden function is the one every caller reaches."""
    m = types.ModuleType("oracle_mutant")
    m.__dict__.update(O.__dict__)
    for name, fn in list(O.__dict__.items()):
        if isinstance(fn, types.FunctionType):
            m.__dict__[name] = types.FunctionType(fn.__code__, m.__dict__, name, fn.__defaults__)
    methods = {}
    for name, fn in O.PaddedBatch.__dict__.items():
        if isinstance(fn, types.FunctionType):
            methods[name] = types.FunctionType(fn.__code__, m.__dict__, name, fn.__defaults__)
    cls = type("PaddedBatch", (O.PaddedBatch,), methods)
    m.PaddedBatch = cls
    for name, fn in overrides.items():
        if name.startswith("PB_"):
            setattr(cls, name[3:], fn)
        else:
            setattr(m, name, fn)
    return m


def _attend_no_scale(q, K, V, scale):
    s = K @ q
    w = np.exp(s - s.max())
    return (w @ V) / w.sum()


def _attend_kv_swapped(q, K, V, scale):
    return O.attend(q, V, K, scale)


def _attend_no_exp(q, K, V, scale):
    s = (K @ q) * scale
    w = s - s.min() + 1e-3
    return (w @ V) / w.sum()


def _attend_unnormalised(q, K, V, scale):
    s = (K @ q) * scale
    w = np.exp(s - s.max())
    return w @ V


def _attend_drop_last(q, K, V, scale):
    return O.attend(q, K[:-1] if len(K) > 1 else K, V[:-1] if len(V) > 1 else V, scale)


def _mask_no_current_column(L, lens):
    M = np.zeros((len(lens), L + 1), np.uint8)
    for b, n in enumerate(lens):
        if n > 0:
            M[b, L - n:L] = 1
    return M


def _mask_start_aligned(L, lens):
    M = np.zeros((len(lens), L + 1), np.uint8)
    for b, n in enumerate(lens):
        if n > 0:
            M[b, :n] = 1
            M[b, L] = 1
    return M


def _pb_mask_no_current_column(self):
    M = O.PaddedBatch.mask(self)
    if not self._shape:
        M[:, -1] = 0
    return M


def _embed_mask_start_aligned(self, slots, lens, k_src, v_src):
    O.PaddedBatch.embed(self, slots, lens, k_src, v_src)
    for s, n in zip(slots, lens):
        self.M[s] = 0
        self.M[s, :n] = 1


def _release_max(self):
    live = self.live()
    r = max(self.L - self.lens[b] for b in live) if live else self.L
    self.K = self.K[:, :, :, r:]
    self.V = self.V[:, :, :, r:]
    self.L -= r
    return r


def _release_none(self):
    return 0


def _embed_start_aligned(self, slots, lens, k_src, v_src):
    O.PaddedBatch.embed(self, slots, lens, k_src, v_src)
    for s, n, ks, vs in zip(slots, lens, k_src, v_src):
        self.K[:, s] = self.fill
        self.V[:, s] = self.fill
        self.K[:, s, :, :n] = ks
        self.V[:, s, :, :n] = vs


def _embed_grow_right(self, slots, lens, k_src, v_src):
    for s, n, ks, vs in zip(slots, lens, k_src, v_src):
        if n > self.L:
            grow = n - self.L
            self.K = np.concatenate([self.K, self._placeholders(grow)], axis=3)
            self.V = np.concatenate([self.V, self._placeholders(grow)], axis=3)
            self.L = n
        self.K[:, s] = self.fill
        self.V[:, s] = self.fill
        self.K[:, s, :, self.L - n:] = ks
        self.V[:, s, :, self.L - n:] = vs
        self.lens[s] = n
        self.hist_k[s] = np.array(ks, copy=True)
        self.hist_v[s] = np.array(vs, copy=True)


def _evict_no_placeholder(self, slots, release=True):
    for s in sorted(slots):
        self.lens[s] = 0
        self.hist_k[s] = self.hist_v[s] = None
    if release:
        self.release()


def _decode_gqa_modulo(self, layer, q, k_new, v_new, scale=None):
    # q-head hq reads kv-head hq % Hkv instead of hq // g
    saved = self.Hq
    out = O.PaddedBatch.decode_layer(self, layer, q, k_new, v_new, scale)
    g = saved // self.Hkv
    if g > 1:
        perm = [(hq % self.Hkv) * g + hq // self.Hkv for hq in range(self.Hq)]
        out = out[:, perm]
    return out


def _decode_prefill_not_causal(self, layer, q, k_new, v_new, scale=None):
    # the new query's positions attend over its whole prompt
    shape = dict(self._shape or {})
    out = O.PaddedBatch.decode_layer(self, layer, q, k_new, v_new, scale)
    sc = 1.0 / np.sqrt(self.D) if scale is None else scale
    g = self.Hq // self.Hkv
    T = self.step_width()
    for b, n in shape.items():
        for t in range(T - n, T):
            for hq in range(self.Hq):
                h = hq // g
                out[b, t, hq] = O.attend(O.widen(q[b, t, hq], self.dtype),
                                         O.widen(k_new[b, T - n:, h], self.dtype),
                                         O.widen(v_new[b, T - n:, h], self.dtype), sc)
    return out


def _mask_padding_in_front(self):
    M = O.PaddedBatch.mask(self)
    if self._shape:
        T = self.step_width()
        for b in range(self.B):
            if b not in self._shape and self.lens[b] > 0:
                M[b, self.L], M[b, self.L + T - 1] = M[b, self.L + T - 1], M[b, self.L]
    return M


def _positions_start_aligned(self, b):
    if self._shape and b in self._shape:
        return list(range(self._shape[b]))
    return [0] if self.lens[b] > 0 else []


def _advance_span_by_one(self):
    T = self.step_width()
    shape = dict(self._shape or {})
    live = [b for b in range(self.B) if self.lens[b] > 0 and b not in shape]
    O.PaddedBatch.advance(self)
    for b in live:
        self.lens[b] -= T - 1


def _widen_bf16_as_fp16(bits, dtype):
    if dtype == O.BF16:
        return np.asarray(bits).astype(np.uint16).view(np.float16).astype(np.float64)
    return O.widen(bits, dtype)


def _widen_shift_15(bits, dtype):
    if dtype == O.BF16:
        return (np.asarray(bits).astype(np.uint32) << np.uint32(15)).view(np.float32).astype(np.float64)
    return O.widen(bits, dtype)


def _widen_flush_subnormals(bits, dtype):
    x = O.widen(bits, dtype)
    return np.where(np.abs(x) < 2.0 ** -126, 0.0 * x, x)


MUTANTS = {
    "scale dropped": dict(attend=_attend_no_scale),
    "keys and values swapped": dict(attend=_attend_kv_swapped),
    "softmax without exp": dict(attend=_attend_no_exp),
    "softmax not normalised": dict(attend=_attend_unnormalised),
    "current token skipped": dict(attend=_attend_drop_last),
    "mask without current column": dict(build_mask=_mask_no_current_column),
    "mask start-aligned": dict(build_mask=_mask_start_aligned),
    "stateful mask without current column": dict(PB_mask=_pb_mask_no_current_column),
    "stateful mask start-aligned": dict(PB_embed=_embed_mask_start_aligned),
    "release takes max": dict(PB_release=_release_max),
    "release never drops": dict(PB_release=_release_none),
    "embed start-aligned": dict(PB_embed=_embed_start_aligned),
    "growth on the right": dict(PB_embed=_embed_grow_right),
    "evicted row keeps its values": dict(PB_evict=_evict_no_placeholder),
    "GQA heads interleaved": dict(PB_decode_layer=_decode_gqa_modulo),
    "prefill not causal": dict(PB_decode_layer=_decode_prefill_not_causal),
    "padding in front of the latest token": dict(PB_mask=_mask_padding_in_front),
    "shorter prompt start-aligned": dict(PB__positions=_positions_start_aligned),
    "span grows by one in a prefill step": dict(PB_advance=_advance_span_by_one),
    "bf16 bits read as fp16": dict(widen=_widen_bf16_as_fp16),
    "bf16 widened by a 15-bit shift": dict(widen=_widen_shift_15),
    "subnormals flushed to zero": dict(widen=_widen_flush_subnormals),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name):
    M = _mutant(**MUTANTS[name])
    caught = []
    for pin in P.ALL_PINS:
        try:
            pin(M)
        except Exception:       # an assertion, or the mutant breaking the pin's own steps
            caught.append(pin.__name__)
    assert caught, f"no pin notices: {name}"
