"""BatonCache: one libbaton handle plus the device buffers it works on.

PyTorch provides device memory and the stream; every operation is one call of
the C ABI (paper_2410_18701_amd/baton.py).
"""
from . import baton as B

_DTYPE_CODE = {"f32": B.BATON_F32, "bf16": B.BATON_BF16}
_FILL = {"f32": B.BATON_FILL_NEG_INF_F32, "bf16": B.BATON_FILL_NEG_INF_BF16}


def torch_dtype(dtype):
    import torch
    return torch.float32 if dtype == "f32" else torch.bfloat16


def _cur_stream():
    import torch
    return torch.cuda.current_stream().cuda_stream


class BatonCache:
    """A batch of `batch` slots over a K/V ring of `capacity` columns per row.

    k, v: [n_layers][batch][n_kv_heads][capacity][head_dim] device tensors,
    each layer dense.  Unless given, they are made with layout "by_layer" --
    views of one [n_layers][2][batch][n_kv_heads][capacity][head_dim] tensor,
    K and V of a layer next to each other (the library streams them about 4%
    faster than from two allocations) -- or "separate" (two tensors).
    """

    def __init__(self, n_layers, batch, n_q_heads, n_kv_heads, head_dim, capacity, dtype="bf16",
                 fill_bits=None, device="cuda", k=None, v=None, assume_filled=False, layout="by_layer"):
        import torch
        self.dtype = dtype
        self.n_layers, self.batch = n_layers, batch
        self.n_q_heads, self.n_kv_heads, self.head_dim = n_q_heads, n_kv_heads, head_dim
        self.capacity = capacity
        self.fill_bits = _FILL[dtype] if fill_bits is None else fill_bits
        tdt = torch_dtype(dtype)
        shape = (n_layers, batch, n_kv_heads, capacity, head_dim)
        if (k is None) != (v is None):
            raise ValueError("give both k and v, or neither")
        if k is None:
            if layout == "by_layer":
                kv = torch.empty((n_layers, 2) + shape[1:], dtype=tdt, device=device)
                k, v = kv[:, 0], kv[:, 1]
            elif layout == "separate":
                k = torch.empty(shape, dtype=tdt, device=device)
                v = torch.empty(shape, dtype=tdt, device=device)
            else:
                raise ValueError(f"unknown layout {layout!r}")
        for name, t in (("k", k), ("v", v)):
            if tuple(t.shape) != shape or t.dtype != tdt or not t[0].is_contiguous():
                raise ValueError(f"{name}: expected {shape} {tdt} with each layer dense")
        if k.stride(0) != v.stride(0):
            raise ValueError("k and v need the same layer stride")
        self.k, self.v = k, v
        desc = B.baton_cache_desc(_DTYPE_CODE[dtype], n_layers, batch, n_q_heads, n_kv_heads,
                                  head_dim, capacity, self.k.data_ptr(), self.v.data_ptr(),
                                  self.fill_bits, self.k.stride(0))
        flags = B.BATON_CREATE_ASSUME_FILLED if assume_filled else 0
        self.handle = B.baton_cache_create(desc, flags, _cur_stream())
        self._ws = None
        self.step_width = 1   # input positions per row of the next step

    # -- workspace --
    def workspace(self):
        import torch
        need = B.baton_decode_attn_workspace_bytes(self.handle)
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(need, dtype=torch.uint8, device=self.k.device)
        return self._ws

    def set_split_tokens(self, tokens):
        B.baton_set_split_tokens(self.handle, tokens)

    # -- the step --
    def evict(self, slots, release=True, scrub=True, stream=None):
        """Finished queries leave; scrub: their tokens become placeholders (else
        they stay as stale bytes the mask excludes); release: drop the leading
        columns that are placeholders in every live row."""
        flags = (B.BATON_RELEASE if release else 0) | (B.BATON_SCRUB if scrub else 0)
        B.baton_kv_evict(self.handle, slots, flags, stream if stream is not None else _cur_stream())

    def embed(self, slots, lens, k_src, v_src, stream=None):
        B.baton_kv_embed(self.handle, slots, lens, k_src, v_src,
                         stream if stream is not None else _cur_stream())

    def move(self, src, dst, stream=None):
        """Live queries src[i] move to free slots dst[i] (cache and mask rows)."""
        B.baton_kv_move(self.handle, src, dst, stream if stream is not None else _cur_stream())

    def shape_insert(self, slots, lens):
        """Prefill these queries inside the batch in the next step (no prefill/decode
        separation); that step's inputs and outputs have a position axis of
        max(lens) after the batch axis."""
        B.baton_shape_insert(self.handle, slots, lens)
        self.step_width = max(int(x) for x in lens)

    def tokens(self):
        """Per-slot token counts (spans without holes)."""
        return B.baton_cache_tokens(self.handle, self.batch)

    def extract(self, slots, stream=None):
        """The slots' cached K and V as new device tensors [n_layers][n_kv_heads][len][head_dim]."""
        import torch
        lens = self.tokens()
        ks, vs = [], []
        for s in slots:
            shape = (self.n_layers, self.n_kv_heads, max(lens[s], 0), self.head_dim)
            ks.append(torch.empty(shape, dtype=self.k.dtype, device=self.k.device))
            vs.append(torch.empty(shape, dtype=self.k.dtype, device=self.k.device))
        B.baton_kv_extract(self.handle, slots, ks, vs, stream if stream is not None else _cur_stream())
        return ks, vs

    def build_mask(self, out=None, stream=None):
        import torch
        L = self.query()[0]
        if out is None:
            out = torch.empty((self.batch, L + self.step_width), dtype=torch.uint8, device=self.k.device)
        B.baton_build_mask(self.handle, out, out.stride(0), stream if stream is not None else _cur_stream())
        return out

    def decode_attn(self, layer, q, k_new, v_new, out=None, scale=0.0, stream=None):
        """q, out: [batch][n_q_heads][head_dim] ([batch][T][...] in a prefill step);
        k_new, v_new: the same with n_kv_heads."""
        import torch
        if out is None:
            out = torch.empty_like(q)
        T = self.step_width
        want_q = self.batch * T * self.n_q_heads * self.head_dim
        want_kv = self.batch * T * self.n_kv_heads * self.head_dim
        for name, t, n in (("q", q, want_q), ("k_new", k_new, want_kv), ("v_new", v_new, want_kv),
                           ("out", out, want_q)):
            if t.dtype != self.k.dtype or not t.is_contiguous() or t.numel() != n:
                raise ValueError(f"{name}: expected {n} contiguous {self.k.dtype} elements, "
                                 f"got {t.numel()} {t.dtype}")
        ws = self.workspace()
        B.baton_decode_attn(self.handle, layer, q, k_new, v_new, out, scale, ws, ws.numel(),
                            stream if stream is not None else _cur_stream())
        return out

    def flush(self, stream=None):
        """Enqueue the placeholder writes evictions still owe."""
        B.baton_cache_flush(self.handle, stream if stream is not None else _cur_stream())

    def advance(self):
        B.baton_step_advance(self.handle)
        self.step_width = 1

    def query(self):
        """(L, base, lens)."""
        return B.baton_cache_query(self.handle, self.batch)

    def logical(self, which="k"):
        """The aligned cache [layer][batch][head][L][dim] read off the ring (a copy)."""
        import torch
        L, base, _ = self.query()
        buf = self.k if which == "k" else self.v
        idx = (torch.arange(L, device=buf.device) + base) % self.capacity
        return buf.index_select(3, idx)

    def close(self):
        if self.handle:
            B.baton_cache_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
