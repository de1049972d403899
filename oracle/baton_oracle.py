"""CPU oracle of Baton's re-batched decode step -- TEST INFRASTRUCTURE ONLY.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import
or run this module.  The library under paper_2410_18701_amd/ never does: the
oracle shares no code with it and exists to check it.

What it computes (Cong et al., "Baton: Enhancing Batch-wise Inference
Efficiency for Large Language Models via Dynamic Re-batching", 2024):

* The batch keeps one dimension-aligned KV_Cache, [layer][batch][head][seq][dim]
  for keys and again for values (sec. 4.1, "Vector Shaping", KV_Cache
  paragraph), and a 0-1 attention_mask [batch][seq+1] (sec. 2.1, "Batch-wise
  inference"; sec. 4.1, second iteration).
* A finished query's slot is reused: its cached keys/values become the
  placeholder value (-inf in the paper) and its mask row becomes 0 (sec. 4.1,
  Attention_mask and KV_Cache paragraphs).
* Leading columns that are placeholders in every live row, [0 : min(index_i)]
  with index_i the end of row i's padding, are released (sec. 4.1, "Resources
  releasing").
* A prefilled query's keys/values are embedded end-aligned into its slot, the
  front filled with placeholders; when the query is longer than the cache, the
  cache first grows on the left, placeholders in the other rows (sec. 4.2,
  "Vector Embedding", the two cases l_q <= l_kv and l_q > l_kv).
* A decode step appends one column of keys/values and one mask column of 1s
  (sec. 4.1, second iteration), and every query attends over its own tokens:
  dot products with the keys, scaling, softmax, weighted sum of the values
  (sec. 2.1, "General architecture").
* The paper's correctness claim: shaping, padding and placeholders do not change
  any query's result (sec. 4.1, the paragraphs closing the insertion example).
* Without prefill/decode separation (sec. 4.1, the Input_token, Attention_mask
  and KV_Cache paragraphs of the insertion example), a new query is prefilled
  inside the batch: the step's input has T = l_q positions per row, the other
  queries' latest token padded behind to T; their mask rows keep their old
  values, 1 for the latest token, 0 for the padding; the new query's row is 0
  over the old columns and 1 over its own tokens; the cache grows by T columns,
  and the padding columns stay in the other rows as holes that are never
  attended to.

Two formulations are kept and must agree: the padded batch (PaddedBatch, the
paper's tensors) and each query's own unpadded history (hist_k / hist_v);
decode_layer returns the result computed from the histories by the plain
definition (attend), in float64 from the exactly widened stored inputs.

Readings where the paper is silent or loose (each listed with its reason in
the design notes of the repository):
* placeholder value: -inf bits by default, any bit pattern allowed; positions
  that hold placeholders are skipped, never multiplied by 0;
* release takes the minimum over live rows only, and an all-free batch has
  length 0;
* l_q == l_kv does not grow the cache;
* the mask has L+1 columns (the current token last), uint8 0/1; free rows are 0;
* a free row's output is 0;
* scale defaults to 1/sqrt(head_dim);
* grouped-query attention maps q-head hq to kv-head hq // (n_q_heads // n_kv_heads);
* several evictions/insertions in one step: evictions (ascending), release,
  then insertions in the given order;
* in-batch prefill of several queries in one step: T = the longest of them,
  a shorter prompt sits at the end of the T new columns with zeros in front
  (the batch's left padding of prompts, sec. 2.1); outputs at positions that
  hold no token are not defined (NaN here), except that a free row's first
  position is 0 as in a decode step; the padding columns hold placeholders;
* a row's length (lens) is its span: columns from its first token to the end
  of the cache, holes included; release drops [0 : min over live rows of the
  first token column].
"""
import math

import numpy as np

F32, BF16 = "f32", "bf16"
STORAGE = {F32: np.uint32, BF16: np.uint16}
NEG_INF_BITS = {F32: 0xFF800000, BF16: 0xFF80}


# ----------------------------------------------------------------- numbers --
def widen(bits, dtype):
    """Stored bits (uint32 fp32 / uint16 bf16) -> float64, exactly.  A bf16
    value is the upper half of the fp32 word with the same bits (sign, 8
    exponent bits, 7 mantissa bits), so its widening is a 16-bit shift."""
    bits = np.asarray(bits)
    if dtype == BF16:
        return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return bits.astype(np.uint32).view(np.float32).astype(np.float64)


def attend(q, K, V, scale):
    """One query's attention over its own tokens (sec. 2.1): softmax(scale * K q) . V.

    q: [D], K and V: [n, D] float64 with n >= 1.  Returns [D] float64.  The max is
    subtracted before exp; that changes no value of the softmax.
    """
    s = (K @ q) * scale
    w = np.exp(s - s.max())
    return (w @ V) / w.sum()


def attend_masked(q, K_row, V_row, mask_row, scale):
    """The same attention read off a padded, aligned row: columns whose mask is 0
    are skipped, so placeholder bits never enter the arithmetic."""
    keep = np.asarray(mask_row).astype(bool)
    return attend(q, K_row[keep], V_row[keep], scale)


def build_mask(L, lens):
    """0-1 mask [batch][L+1]: row b is 1 on its last lens[b] cached columns and on
    column L (the current token) when the slot is live, all 0 when it is free."""
    M = np.zeros((len(lens), L + 1), dtype=np.uint8)
    for b, n in enumerate(lens):
        if n > 0:
            M[b, L - n:] = 1
    return M


def expected_row_masked(mask_row, hist_row, fill_bits, dtype):
    """A row of the aligned cache whose tokens sit where mask_row (its cached
    columns) is 1, in order; placeholders elsewhere."""
    keep = np.asarray(mask_row).astype(bool)
    hist_row = np.asarray(hist_row)
    out = np.full((len(keep), hist_row.shape[-1]), fill_bits, dtype=STORAGE[dtype])
    out[keep] = hist_row
    return out


# ------------------------------------------------------------ padded batch --
class PaddedBatch:
    """The paper's batch: aligned KV_Cache + attention_mask + per-query histories.

    K, V: [n_layers][batch][n_kv_heads][L][head_dim] stored bits.  With
    materialize=False only the lengths are tracked -- no tensors, no histories --
    for large workloads whose rows are checked one at a time against histories
    rebuilt from the input generator, with attend.
    """

    def __init__(self, n_layers, batch, n_q_heads, n_kv_heads, head_dim, dtype,
                 fill_bits=None, materialize=True):
        if n_q_heads % n_kv_heads:
            raise ValueError("n_q_heads must be a multiple of n_kv_heads")
        self.NL, self.B, self.Hq, self.Hkv, self.D = n_layers, batch, n_q_heads, n_kv_heads, head_dim
        self.dtype = dtype
        self.fill = NEG_INF_BITS[dtype] if fill_bits is None else fill_bits
        self.materialize = materialize
        self.L = 0
        self.lens = [0] * batch
        st = STORAGE[dtype]
        shape = (n_layers, batch, n_kv_heads, 0, head_dim)
        self.K = np.zeros(shape, st) if materialize else None
        self.V = np.zeros(shape, st) if materialize else None
        self.hist_k = [None] * batch   # per slot: [layer][head][n][dim] bits of its query
        self.hist_v = [None] * batch
        self.M = np.zeros((batch, 0), np.uint8)   # attention_mask over the cached columns
        self._new_k = None             # columns being appended this step, per layer
        self._new_v = None
        self._layers_done = set()
        self._shape = None             # pending in-batch prefill: {slot: prompt length}

    # -- helpers --
    def _placeholders(self, n_cols, rows=None):
        rows = self.B if rows is None else rows
        return np.full((self.NL, rows, self.Hkv, n_cols, self.D), self.fill, STORAGE[self.dtype])

    def live(self):
        return [b for b in range(self.B) if self.lens[b] > 0]

    def _check_between_steps(self):
        if self._layers_done:
            raise RuntimeError("a decode step is in progress")
        if self._shape is not None:
            raise RuntimeError("an in-batch prefill is registered for the next step")

    def step_width(self):
        """Positions per row in the next step's input: 1, or T with an in-batch prefill."""
        return max(self._shape.values()) if self._shape else 1

    # -- the method's steps --
    def evict(self, slots, release=True):
        """Finished queries leave; their keys/values become placeholders, then the
        shared leading placeholder columns are released."""
        self._check_between_steps()
        slots = sorted(slots)
        if len(set(slots)) != len(slots) or any(not 0 <= s < self.B for s in slots):
            raise ValueError("bad slot list")
        if any(self.lens[s] == 0 for s in slots):
            raise LookupError("evicting a free slot")
        for s in slots:
            if self.materialize:
                self.K[:, s] = self.fill
                self.V[:, s] = self.fill
            self.M[s] = 0
            self.lens[s] = 0
            self.hist_k[s] = self.hist_v[s] = None
        if release:
            self.release()

    def release(self):
        """Drop columns [0 : min_i index_i], index_i = L - len_i over live rows."""
        self._check_between_steps()
        live = self.live()
        r = min(self.L - self.lens[b] for b in live) if live else self.L
        if self.materialize:
            self.K = self.K[:, :, :, r:]
            self.V = self.V[:, :, :, r:]
        self.M = self.M[:, r:]
        self.L -= r
        return r

    def embed(self, slots, lens, k_src, v_src):
        """Insert prefilled queries: k_src[i], v_src[i] are bits [layer][head][lens[i]][dim]."""
        self._check_between_steps()
        if len(set(slots)) != len(slots) or any(not 0 <= s < self.B for s in slots):
            raise ValueError("bad slot list")
        if any(n < 1 for n in lens):
            raise ValueError("a prefilled query has at least one token")
        if any(self.lens[s] != 0 for s in slots):
            raise LookupError("embedding into a live slot")
        for s, n, ks, vs in zip(slots, lens, k_src, v_src):
            if n > self.L:                          # case l_q > l_kv: grow on the left
                grow = n - self.L
                if self.materialize:
                    self.K = np.concatenate([self._placeholders(grow), self.K], axis=3)
                    self.V = np.concatenate([self._placeholders(grow), self.V], axis=3)
                self.M = np.concatenate([np.zeros((self.B, grow), np.uint8), self.M], axis=1)
                self.L = n
            self.M[s] = 0
            self.M[s, self.L - n:] = 1
            if self.materialize:                    # case l_q <= l_kv: end-aligned
                self.K[:, s] = self.fill
                self.V[:, s] = self.fill
                self.K[:, s, :, self.L - n:] = ks
                self.V[:, s, :, self.L - n:] = vs
            self.lens[s] = n
            if self.materialize:
                self.hist_k[s] = np.array(ks, copy=True)
                self.hist_v[s] = np.array(vs, copy=True)

    def extract(self, slots):
        """A live query's keys and values read off its aligned row (the columns
        after its placeholders), to be stored aside and re-embedded later
        (sec. 4.3, preemptive scheduling and batch-size scaling).  Changes nothing."""
        self._check_between_steps()
        if len(set(slots)) != len(slots) or any(not 0 <= s < self.B for s in slots):
            raise ValueError("bad slot list")
        if any(self.lens[s] == 0 for s in slots):
            raise LookupError("extracting a free slot")
        out = []
        for s in slots:
            keep = self.M[s].astype(bool)
            out.append((self.K[:, s][:, :, keep].copy(), self.V[:, s][:, :, keep].copy()))
        return out

    def move(self, src, dst):
        """Live queries change slots: query src[i] moves, cache and mask row bit
        for bit, into the free slot dst[i], which leaves src[i] free -- moving
        queries within the batch (sec. 4.3), e.g. to gather the live rows at
        the front of the batch dimension.  L does not change."""
        self._check_between_steps()
        if len(src) != len(dst) or len(set(src) | set(dst)) != 2 * len(src) or \
                any(not 0 <= s < self.B for s in list(src) + list(dst)):
            raise ValueError("bad slot lists")
        if any(self.lens[s] == 0 for s in src) or any(self.lens[d] != 0 for d in dst):
            raise LookupError("moving a free slot or into a live one")
        for s, d in zip(src, dst):
            if self.materialize:
                self.K[:, d] = self.K[:, s]
                self.V[:, d] = self.V[:, s]
                self.K[:, s] = self.fill
                self.V[:, s] = self.fill
            self.M[d] = self.M[s]
            self.M[s] = 0
            self.lens[d], self.lens[s] = self.lens[s], 0
            self.hist_k[d], self.hist_v[d] = self.hist_k[s], self.hist_v[s]
            self.hist_k[s] = self.hist_v[s] = None

    def shape_insert(self, slots, lens):
        """Register new queries to be prefilled inside the batch in the next step
        (no prefill/decode separation, sec. 4.1): slots must be free, lens are
        their prompt lengths.  The step's input then has T = max(lens) positions
        per row."""
        self._check_between_steps()
        if not slots or len(set(slots)) != len(slots) or any(not 0 <= s < self.B for s in slots):
            raise ValueError("bad slot list")
        if len(lens) != len(slots) or any(n < 1 for n in lens):
            raise ValueError("a prompt has at least one token")
        if any(self.lens[s] != 0 for s in slots):
            raise LookupError("shaping into a live slot")
        self._shape = {s: int(n) for s, n in zip(slots, lens)}

    def mask(self):
        """attention_mask of the next step: the cached columns, then the step's
        own input columns (one, or T with an in-batch prefill)."""
        if not self._shape:
            cur = np.array([[1 if n > 0 else 0] for n in self.lens], np.uint8).reshape(self.B, 1)
            return np.concatenate([self.M, cur], axis=1)
        T = self.step_width()
        M = np.zeros((self.B, self.L + T), np.uint8)
        for b in range(self.B):
            if b in self._shape:                 # old columns 0, its own tokens 1
                M[b, self.L + T - self._shape[b]:] = 1
            elif self.lens[b] > 0:               # old values, latest token 1, padding 0
                M[b, :self.L] = self.M[b]
                M[b, self.L] = 1
        return M

    def _positions(self, b):
        """Input positions of row b that hold a token in the next step."""
        T = self.step_width()
        if self._shape and b in self._shape:
            return list(range(T - self._shape[b], T))
        return [0] if self.lens[b] > 0 else []

    def decode_layer(self, layer, q, k_new, v_new, scale=None):
        """One layer of the step.

        Decode step: q bits [batch][n_q_heads][dim]; k_new, v_new bits
        [batch][n_kv_heads][dim].  With an in-batch prefill registered, every
        input has a position axis after the batch: [batch][T][...][dim].
        Appends this layer's new columns (placeholders where no token is) and
        returns the attention output float64 in q's shape, computed from each
        query's own tokens: 0 for a free row's first position, NaN at positions
        that hold no token.
        """
        if layer in self._layers_done:
            raise RuntimeError("layer already decoded this step")
        if not self.materialize:
            self._layers_done.add(layer)
            return None
        scale = 1.0 / math.sqrt(self.D) if scale is None else scale
        st = STORAGE[self.dtype]
        T = self.step_width()
        shaped = self._shape is not None
        if not shaped:                           # one position: add the axis
            q, k_new, v_new = q[:, None], k_new[:, None], v_new[:, None]
        if q.shape[1] != T or k_new.shape[1] != T or v_new.shape[1] != T:
            raise ValueError("inputs must have one position per column of the step")
        if self._new_k is None:
            self._new_k = np.full((self.NL, self.B, self.Hkv, T, self.D), self.fill, st)
            self._new_v = np.full((self.NL, self.B, self.Hkv, T, self.D), self.fill, st)
        g = self.Hq // self.Hkv
        out = np.full((self.B, T, self.Hq, self.D), np.nan)
        for b in range(self.B):
            pos = self._positions(b)
            if not pos:
                out[b, 0] = 0.0
                continue
            for t in pos:
                self._new_k[layer, b, :, t] = k_new[b, t]
                self._new_v[layer, b, :, t] = v_new[b, t]
            for t in pos:
                for hq in range(self.Hq):
                    h = hq // g
                    if shaped and b in self._shape:      # the new query: its prompt up to t
                        K = widen(k_new[b, pos[0]:t + 1, h], self.dtype)
                        V = widen(v_new[b, pos[0]:t + 1, h], self.dtype)
                    else:                                # its history and the latest token
                        K = widen(np.concatenate([self.hist_k[b][layer, h], k_new[b, t, h][None]]), self.dtype)
                        V = widen(np.concatenate([self.hist_v[b][layer, h], v_new[b, t, h][None]]), self.dtype)
                    out[b, t, hq] = attend(widen(q[b, t, hq], self.dtype), K, V, scale)
        self._layers_done.add(layer)
        return out if shaped else out[:, 0]

    def decode_layer_padded(self, layer, q, scale=None):
        """The batched formulation of the same layer: masked attention over the
        padded rows (after decode_layer appended this layer's columns); the query
        at input position t sees the mask's columns up to L + t."""
        if layer not in self._layers_done or not self.materialize:
            raise RuntimeError("decode_layer first, on a materialized batch")
        scale = 1.0 / math.sqrt(self.D) if scale is None else scale
        shaped = self._shape is not None
        if not shaped:
            q = q[:, None]
        T = self.step_width()
        g = self.Hq // self.Hkv
        M = self.mask()
        K = np.concatenate([self.K[layer], self._new_k[layer]], axis=2)
        V = np.concatenate([self.V[layer], self._new_v[layer]], axis=2)
        out = np.full((self.B, T, self.Hq, self.D), np.nan)
        for b in range(self.B):
            pos = self._positions(b)
            if not pos:
                out[b, 0] = 0.0
            for t in pos:
                c = self.L + t + 1
                for hq in range(self.Hq):
                    h = hq // g
                    out[b, t, hq] = attend_masked(widen(q[b, t, hq], self.dtype),
                                                  widen(K[b, h, :c], self.dtype),
                                                  widen(V[b, h, :c], self.dtype), M[b, :c], scale)
        return out if shaped else out[:, 0]

    def advance(self):
        """Close the step: every layer appended its columns; the mask takes the
        step's columns; rows that decoded grow by one token."""
        if len(self._layers_done) != self.NL:
            raise RuntimeError("every layer must be decoded before the step advances")
        T = self.step_width()
        M_step = self.mask()[:, self.L:]
        if self.materialize:
            self.K = np.concatenate([self.K, self._new_k], axis=3)
            self.V = np.concatenate([self.V, self._new_v], axis=3)
        for b in range(self.B):
            pos = self._positions(b)
            if not pos:
                continue
            if self.materialize:
                k_tok = self._new_k[:, b][:, :, pos]
                v_tok = self._new_v[:, b][:, :, pos]
                if self._shape and b in self._shape:
                    self.hist_k[b], self.hist_v[b] = k_tok, v_tok
                else:
                    self.hist_k[b] = np.concatenate([self.hist_k[b], k_tok], axis=2)
                    self.hist_v[b] = np.concatenate([self.hist_v[b], v_tok], axis=2)
            if self._shape and b in self._shape:
                self.lens[b] = self._shape[b]
            else:
                self.lens[b] += T
        self.M = np.concatenate([self.M, M_step], axis=1)
        self.L += T
        self._new_k = self._new_v = None
        self._layers_done = set()
        self._shape = None
