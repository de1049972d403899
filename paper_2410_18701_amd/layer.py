"""A whole decode layer around the re-batched attention, as C-ABI calls.

Each method is argument marshalling for one libbaton call (paper_2410_18701_amd/
baton.py); PyTorch provides the buffers.  The layer is the paper's model's
(llama2-7b, sec. 5): RMS norm -> fused QKV projection -> rotary embedding at
each query's token count -> re-batched attention (BatonCache.decode_attn) ->
output projection added to the residual stream -> RMS norm -> gate/up
projection -> silu(gate) * up -> down projection added to the residual stream.
"""
from . import baton as B


def _stream():
    import torch
    return torch.cuda.current_stream().cuda_stream


class PackedWeight:
    """A weight in the packed form baton_linear_packed reads."""

    def __init__(self, data, out_dim, in_dim):
        self.data, self.out_dim, self.in_dim = data, out_dim, in_dim


class Gemm:
    """The device workspace of the projections (the partial sums of
    baton_linear_packed when it splits along in_dim), and the projection calls."""

    def __init__(self, ws_bytes=32 << 20):
        import torch
        self.ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda") if ws_bytes else None
        self.ws_bytes = ws_bytes

    def pack(self, w):
        """The packed form of a weight w [out][in] for linear_packed (made once per weight)."""
        import torch
        out_dim, in_dim = w.shape
        if not w.is_contiguous():
            raise ValueError("pack: contiguous tensors only")
        wp = torch.empty(B.baton_linear_packed_bytes(out_dim, in_dim) // 2, dtype=w.dtype, device=w.device)
        B.baton_linear_pack(B.BATON_BF16, w, wp, out_dim, in_dim, _stream())
        return PackedWeight(wp, out_dim, in_dim)

    def linear_packed(self, x, wp, y, accumulate=False):
        """y (+)= x . w^T with w packed by pack(); x [rows <= 256][in], y [rows][out]."""
        rows, in_dim = x.shape
        if in_dim != wp.in_dim or tuple(y.shape) != (rows, wp.out_dim):
            raise ValueError("linear_packed: shapes do not match")
        for t in (x, y):
            if not t.is_contiguous():
                raise ValueError("linear_packed: contiguous tensors only")
        B.baton_linear_packed(B.BATON_BF16, x, wp.data, y, rows, wp.out_dim, in_dim, accumulate, self.ws,
                              self.ws_bytes, _stream())
        return y

    def linear_packed_silu(self, x, wp, out):
        """out = silu(x . gate^T) * (x . up^T) for the packed [gate; up] weight wp
        (bit for bit linear_packed unsplit, then silu_mul, in one kernel)."""
        rows, in_dim = x.shape
        if in_dim != wp.in_dim or tuple(out.shape) != (rows, wp.out_dim // 2):
            raise ValueError("linear_packed_silu: shapes do not match")
        for t in (x, out):
            if not t.is_contiguous():
                raise ValueError("linear_packed_silu: contiguous tensors only")
        B.baton_linear_packed_silu(B.BATON_BF16, x, wp.data, out, rows, wp.out_dim, in_dim, _stream())
        return out

    def linear_packed_rmsnorm(self, x, wp, y, gain, eps, y_norm, accumulate=False):
        """linear_packed, then y_norm = rmsnorm(y, gain, eps) (bit for bit; one
        kernel adds the split sums and normalises when the product splits)."""
        rows, in_dim = x.shape
        if in_dim != wp.in_dim or tuple(y.shape) != (rows, wp.out_dim) or tuple(y_norm.shape) != tuple(y.shape) \
                or gain.numel() != wp.out_dim:
            raise ValueError("linear_packed_rmsnorm: shapes do not match")
        for t in (x, y, y_norm, gain):
            if not t.is_contiguous():
                raise ValueError("linear_packed_rmsnorm: contiguous tensors only")
        B.baton_linear_packed_rmsnorm(B.BATON_BF16, x, wp.data, y, rows, wp.out_dim, in_dim, accumulate, gain,
                                      eps, y_norm, self.ws, self.ws_bytes, _stream())
        return y

    def close(self):
        self.ws = None


def rmsnorm(x, gain, y, eps):
    rows, dim = x.shape
    if tuple(y.shape) != (rows, dim) or gain.numel() != dim:
        raise ValueError("rmsnorm: shapes do not match")
    B.baton_rmsnorm(B.BATON_BF16, x, gain, y, rows, dim, eps, _stream())
    return y


def silu_mul(gate_up, out):
    rows, two_f = gate_up.shape
    if tuple(out.shape) != (rows, two_f // 2):
        raise ValueError("silu_mul: shapes do not match")
    B.baton_silu_mul(B.BATON_BF16, gate_up, out, rows, two_f // 2, _stream())
    return out


def rope_qkv(cache, qkv, q, k_new, v_new, theta):
    width = (cache.n_q_heads + 2 * cache.n_kv_heads) * cache.head_dim
    if tuple(qkv.shape) != (cache.batch, width):
        raise ValueError("rope_qkv: qkv must be [batch][(Hq + 2 Hkv) * head_dim]")
    if q.numel() != cache.batch * cache.n_q_heads * cache.head_dim or \
            k_new.numel() != cache.batch * cache.n_kv_heads * cache.head_dim or v_new.numel() != k_new.numel():
        raise ValueError("rope_qkv: output sizes do not match the cache")
    B.baton_rope_qkv(cache.handle, qkv, q, k_new, v_new, theta, _stream())


class DecodeLayers:
    """The layers of one model over one BatonCache, with preallocated activations.

    weights[layer]: dict of bf16 device tensors norm1 [hid], qkv [(Hq + 2 Hkv) D][hid],
    o [hid][Hq D], norm2 [hid], gate_up [2 F][hid], down [hid][F].  The projections
    run on the weight-streaming GEMM over packed copies of the weights, made here
    once.  Each residual add is fused with the normalisation that follows it (the
    output projection with norm2, the down projection with the next layer's
    norm1), so layer(l + 1) expects x as layer(l) returned it, and the gate/up
    projection with the gated activation."""

    PROJ = ("qkv", "o", "gate_up", "down")

    def __init__(self, cache, weights, gemm, theta=10000.0, eps=1e-5):
        import torch
        self.cache, self.w, self.gemm, self.theta, self.eps = cache, weights, gemm, theta, eps
        Bt, Hq, Hkv, D = cache.batch, cache.n_q_heads, cache.n_kv_heads, cache.head_dim
        if Bt > B.BATON_GEMM_MAX_ROWS:
            raise ValueError(f"at most {B.BATON_GEMM_MAX_ROWS} slots")
        self.wp = [{k: gemm.pack(w[k]) for k in self.PROJ} for w in weights]
        hid = weights[0]["norm1"].numel()
        F = weights[0]["down"].shape[1]
        e = lambda *s: torch.empty(s, dtype=torch.bfloat16, device="cuda")
        self.h, self.qkv = e(Bt, hid), e(Bt, (Hq + 2 * Hkv) * D)
        self.q, self.k, self.v, self.att = e(Bt, Hq, D), e(Bt, Hkv, D), e(Bt, Hkv, D), e(Bt, Hq, D)
        self.gu, self.act = e(Bt, 2 * F), e(Bt, F)
        self._normed = None   # (layer, x) whose norm1 input h already holds

    def layer(self, layer, x):
        """One layer of the decode step on the residual stream x [batch][hid] (in place)."""
        w, wp, g = self.w[layer], self.wp[layer], self.gemm
        if self._normed != (layer, x.data_ptr()):   # h holds norm1(x) after the previous layer
            rmsnorm(x, w["norm1"], self.h, self.eps)
        self._normed = None
        g.linear_packed(self.h, wp["qkv"], self.qkv)
        rope_qkv(self.cache, self.qkv, self.q, self.k, self.v, self.theta)
        self.cache.decode_attn(layer, self.q, self.k, self.v, out=self.att)
        att = self.att.view(self.att.shape[0], -1)
        g.linear_packed_rmsnorm(att, wp["o"], x, w["norm2"], self.eps, self.h, accumulate=True)
        if wp["gate_up"].out_dim % 32 == 0:
            g.linear_packed_silu(self.h, wp["gate_up"], self.act)
        else:
            g.linear_packed(self.h, wp["gate_up"], self.gu)
            silu_mul(self.gu, self.act)
        if layer + 1 < len(self.w):
            g.linear_packed_rmsnorm(self.act, wp["down"], x, self.w[layer + 1]["norm1"], self.eps, self.h,
                                    accumulate=True)
            self._normed = (layer + 1, x.data_ptr())
        else:
            g.linear_packed(self.act, wp["down"], x, accumulate=True)
        return x
