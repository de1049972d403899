/*
 * baton.h -- C ABI of libbaton.so: the re-batched decode step of Baton
 * (Cong, Chen, Zhao, Yang, "Baton: Enhancing Batch-wise Inference Efficiency
 * for Large Language Models via Dynamic Re-batching", 2024) on MI355X (gfx950).
 *
 * One batch of `batch` slots decodes together over a dimension-aligned KV cache
 * (sec. 4.1, "Vector Shaping"): every row (layer, slot, kv-head) has the same
 * padded length L, a live slot's tokens sit at the right end of its row
 * (columns L-len .. L-1) and everything before them is a placeholder.  Between
 * decode steps, finished queries leave (baton_kv_evict) and prefilled queries
 * take free slots (baton_kv_embed, sec. 4.2, "Vector Embedding"); each step
 * then runs masked attention for one new token per query (baton_decode_attn)
 * and appends that token's key/value as column L (sec. 4.1, second iteration).
 *
 * Without prefill/decode separation (sec. 4.1, the Input_token, Attention_mask
 * and KV_Cache paragraphs), a new query is instead prefilled inside the batch
 * (baton_shape_insert): that step's input has T positions per row, T the
 * longest new prompt, the other queries' latest token padded behind to T, and
 * the cache grows by T columns.  The padding columns stay in the other rows as
 * holes: placeholders inside a live row that its mask zeroes and attention
 * skips.  A row's length (its span) then counts the holes between its first
 * token and the end of the cache; baton_cache_tokens gives its token count.
 *
 * Conventions
 *  - Every call returns a baton_status.  Arguments and state are checked on the
 *    host before anything is enqueued; on any error nothing is enqueued and the
 *    cache's state is unchanged.
 *  - Device work is enqueued on the caller's stream and the call returns at
 *    once (stream order, no host synchronisation).  All work on one cache must
 *    go to one stream; a handle is not thread-safe.
 *  - Ownership: the caller allocates and owns all device memory (the K/V ring
 *    buffers, sources, q/k_new/v_new/out, mask, workspace).  The library owns
 *    only the host handle and never allocates device memory.  Device buffers
 *    must stay valid until the stream has passed the call that uses them.
 *  - Element types: fp32 or bf16 storage, fp32 arithmetic.  head_dim 64 or 128;
 *    n_q_heads / n_kv_heads in {1, 2, 4, 8}; batch <= BATON_MAX_BATCH.
 *
 * Memory layout (device).  K and V are each
 *     [n_layers][batch][n_kv_heads][capacity][head_dim]
 * contiguous elements.  The `capacity` columns of a row form a ring: logical
 * column j of the aligned cache (0 <= j < L) lives at physical column
 * (base + j) mod capacity, where base is reported by baton_cache_query.  As
 * long as every eviction since the handle was created asked for BATON_SCRUB,
 * every physical position that is not a live token holds the placeholder bits
 * (fill_bits) -- free rows, the placeholder fronts of live rows and the
 * capacity - L unused columns alike -- except the tokens of slots evicted since
 * the last decode step began, whose placeholder write is deferred (see
 * baton_kv_evict).  An eviction without BATON_SCRUB leaves its query's tokens
 * in place as stale bytes; no kernel ever reads a position that is not a live
 * token, so results do not depend on what such positions hold.
 */
#ifndef BATON_H
#define BATON_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum baton_status {
  BATON_OK = 0,
  BATON_EINVAL = 1,    /* malformed argument: null pointer, size or index out of range, duplicate slot */
  BATON_ESLOT = 2,     /* evicting a free slot, or embedding into a live one */
  BATON_ECAPACITY = 3, /* the padded length plus the next appended columns would exceed capacity,
                          or a prefill step would leave more than BATON_MAX_HOLES holes */
  BATON_EDTYPE = 4,    /* unsupported element type, head_dim or head grouping */
  BATON_ESTATE = 5,    /* call out of order with the decode step in progress */
  BATON_EHIP = 6,      /* the HIP runtime refused a launch */
  BATON_ESCRATCH = 7   /* baton_decode_attn_noalloc: the step needs more than BATON_SCRATCH_BYTES */
} baton_status;

typedef enum baton_dtype { BATON_F32 = 0, BATON_BF16 = 1 } baton_dtype;

/* The paper's placeholder value, -inf (sec. 4.1, KV_Cache paragraph; sec. 4.2). */
#define BATON_FILL_NEG_INF_F32 0xFF800000u
#define BATON_FILL_NEG_INF_BF16 0xFF80u

#define BATON_MAX_BATCH 512
#define BATON_MAX_PREFILL 64 /* queries prefilled inside the batch in one step */
#define BATON_MAX_HOLES 64   /* prefill steps whose padding columns are still inside live rows */

/* baton_cache_create flags */
#define BATON_CREATE_ASSUME_FILLED 1u /* K and V already hold fill_bits everywhere: enqueue nothing */

/* baton_kv_evict flags */
#define BATON_RELEASE 1u /* then release the leading columns that are placeholders in every live row */
#define BATON_SCRUB 2u   /* overwrite the finished queries' tokens with the placeholder */

typedef struct baton_cache_desc {
  int32_t dtype;      /* baton_dtype of K, V, sources, q, k_new, v_new and out */
  int32_t n_layers;   /* >= 1 */
  int32_t batch;      /* slots, 1 .. BATON_MAX_BATCH */
  int32_t n_q_heads;  /* query heads per layer */
  int32_t n_kv_heads; /* key/value heads per layer (n_q_heads / n_kv_heads in {1,2,4,8}) */
  int32_t head_dim;   /* 64 or 128 */
  int64_t capacity;   /* ring columns per row, >= 2 */
  void* k;            /* device, [n_layers][batch][n_kv_heads][capacity][head_dim], 16-byte aligned;
                         layer l's rows (dense) at k + l * layer_stride elements */
  void* v;            /* device, same layout as k */
  uint32_t fill_bits; /* placeholder bit pattern in the low 32 (fp32) or 16 (bf16) bits */
  int64_t layer_stride; /* elements from layer l's rows to layer l + 1's, in k and in v alike;
                           0: packed (batch * n_kv_heads * capacity * head_dim).  A larger
                           stride lets K and V share one allocation interleaved by layer,
                           [n_layers][2][batch][n_kv_heads][capacity][head_dim] (v = k + one
                           layer's rows, layer_stride = two layers' rows): reading a layer's K
                           and V rows close together streams about 4% faster than from two
                           separate allocations.  A whole number of 16-byte vectors; no layer
                           of k may overlap a layer of v. */
} baton_cache_desc;

typedef struct baton_cache baton_cache; /* opaque host handle */

/*
 * Create a handle for an empty batch: L = 0, every slot free.  Unless
 * BATON_CREATE_ASSUME_FILLED is given, enqueues on `stream` the write of
 * fill_bits over all of K and V.  The descriptor is copied.
 * Errors: EINVAL (null out/k/v, sizes out of range, misaligned k/v,
 * layer_stride below one layer's rows or not a whole number of 16-byte
 * vectors, k and v overlapping), EDTYPE (dtype, head_dim or grouping
 * unsupported), EHIP.
 */
baton_status baton_cache_create(const baton_cache_desc* desc, uint32_t flags, hipStream_t stream,
                                baton_cache** out);

/* Free the host handle (device memory stays the caller's).  NULL is accepted. */
baton_status baton_cache_destroy(baton_cache* cache);

/*
 * Finished queries leave their slots (sec. 4.1, Attention_mask and KV_Cache
 * paragraphs: the finished query's mask row is zeroed, which alone keeps its
 * tokens out of every later attention; overwriting its cached keys/values
 * with the placeholder is the further safeguard the paper recommends).
 * slots: host array of n distinct live slot indices (n may be 0); the slots
 * become free.
 * With BATON_SCRUB, the placeholder write over each finished query's tokens
 * (every layer and head; the holes of its row hold placeholders already and
 * are skipped) is owed, not enqueued here: the next baton_kv_embed into the
 * slot performs it over the columns in front of its new query (the new query
 * overwrites the rest), and the first baton_decode_attn of the next step, or
 * baton_cache_flush, performs whatever is still owed.  Without BATON_SCRUB no
 * placeholder byte is written: the tokens stay as stale bytes that the mask
 * excludes and no kernel reads.
 * With BATON_RELEASE, the columns [0 : min over live rows of (L - len)] are
 * then released (sec. 4.1, "Resources releasing"): L becomes the longest live
 * span (0 when no slot is live).  Without it L is unchanged; release is
 * optional and may come with any later eviction (including one of no slot).
 * Release moves no data.  Nothing is enqueued.
 * Errors: EINVAL (n < 0, null slots with n > 0, index out of range, duplicate,
 * unknown flag), ESLOT (a slot is free), ESTATE (inside a decode step).
 */
baton_status baton_kv_evict(baton_cache* cache, const int32_t* slots, int32_t n, uint32_t flags,
                            hipStream_t stream);

/*
 * Prefilled queries take free slots (sec. 4.2, "Vector Embedding").  slots and
 * lens: host arrays of n entries (n may be 0); k_src and v_src: host arrays of
 * n device pointers, each [n_layers][n_kv_heads][lens[i]][head_dim] contiguous,
 * 16-byte aligned.  If the longest query exceeds L (the case l_q > l_kv), the
 * batch first grows on the left to that length, every other row's new front
 * being placeholders; then each query's keys/values are copied end-aligned into
 * its slot, placeholders in front (the case l_q <= l_kv).  Growth moves no
 * data: the new front columns already hold placeholders.  The same launch writes
 * the placeholders an embedded slot still owes from its eviction.
 * Errors: EINVAL (n < 0, null arrays or pointers, slot out of range, duplicate,
 * lens[i] < 1), ESLOT (a slot is live), ECAPACITY (max(L, max lens) + 1 >
 * capacity), ESTATE (inside a decode step), EHIP.
 */
baton_status baton_kv_embed(baton_cache* cache, const int32_t* slots, int32_t n, const int32_t* lens,
                            const void* const* k_src, const void* const* v_src, hipStream_t stream);

/*
 * Copy live queries' cached keys/values out of the batch (sec. 4.3: preemptive
 * scheduling stores the lowest-priority query's keys and values aside and
 * re-inserts it later; batch-size scaling moves queries' keys and values to
 * host memory and back).  slots: host array of n distinct live slots; k_dst,
 * v_dst: host arrays of n device pointers, each receiving
 * [n_layers][n_kv_heads][len][head_dim] contiguous elements (len = the slot's
 * token count, baton_cache_tokens; holes are skipped), 16-byte aligned -- the
 * layout baton_kv_embed takes, so baton_kv_embed(slot', len, k_dst, v_dst)
 * re-inserts the query into any free slot with its tokens bit for bit.  The
 * batch is not changed; preempting a query is extract, then baton_kv_evict.
 * The destinations (and baton_kv_embed's sources) may be device memory or
 * pinned host memory mapped for the device (hipHostMalloc; pass its device
 * address, hipHostGetDevicePointer): the kernel then moves the tokens over the
 * host link directly, with no device staging -- queries parked in host memory
 * to scale the batch.
 * Errors: EINVAL (n < 0, null arrays or pointers, misaligned pointer, slot out
 * of range, duplicate), ESLOT (a slot is free), ESTATE (inside a decode step),
 * EHIP.
 */
baton_status baton_kv_extract(const baton_cache* cache, const int32_t* slots, int32_t n,
                              void* const* k_dst, void* const* v_dst, hipStream_t stream);

/*
 * Live queries change slots (sec. 4.3 moves queries within and out of the
 * batch; moving the live ones to the front compacts the batch dimension):
 * src, dst host arrays of n pairs, src[i] live, dst[i] free, no slot listed
 * twice.  Query src[i]'s row -- its tokens, holes and mask -- moves bit for bit
 * into slot dst[i] (same columns), and src[i] becomes free, its tokens owed
 * placeholders as after an eviction.  L and base do not change.  One launch
 * (plus one for placeholders the targets still owed).
 * Errors: EINVAL (n < 0, null arrays, slot out of range or listed twice),
 * ESLOT (a source free or a target live), ESTATE (inside a decode step, or a
 * prefill registered), EHIP.
 */
baton_status baton_kv_move(baton_cache* cache, const int32_t* src, const int32_t* dst, int32_t n,
                           hipStream_t stream);

/*
 * Prefill new queries inside the batch in the next step (sec. 4.1, without
 * prefill/decode separation).  slots, lens: host arrays of n >= 1 entries:
 * distinct free slots and their prompt lengths.  The next step's input has
 * T = max(lens) positions per row: a new query's prompt at the last lens[i]
 * positions, every other live query's latest token at position 0 and padding
 * behind it.  That step's baton_decode_attn calls take q, k_new, v_new and out
 * with a position axis of T after the batch axis; baton_build_mask returns
 * L + T columns; baton_step_advance then grows L by T, leaves a hole of T - 1
 * columns behind the latest token of every other live row, and makes the new
 * queries live with lens[i] tokens.  Host metadata only; replaces a previous
 * registration for the same step.
 * Errors: EINVAL (n < 1 or > BATON_MAX_PREFILL, null arrays, slot out of range,
 * duplicate, lens[i] < 1), ESLOT (a slot is live), ECAPACITY (L + T >
 * capacity, or more than BATON_MAX_HOLES holes would remain), ESTATE (inside a
 * decode step).
 */
baton_status baton_shape_insert(baton_cache* cache, const int32_t* slots, int32_t n,
                                const int32_t* lens);

/*
 * The 0-1 attention mask of the current step (sec. 2.1, "Batch-wise inference";
 * sec. 4.1: a column of ones for the current token, zero rows for finished
 * queries; sec. 4.2: zeros over the grown front of existing rows).  Writes
 * mask[b * ld + j] for 0 <= j < L + T (T = 1, or the prefill width after
 * baton_shape_insert): for a live slot, 1 on its own tokens' columns and on
 * column L (its token being decoded), 0 on its holes, in front of its first
 * token and after column L; for a slot being prefilled, 1 on its prompt's
 * columns (the last lens[i] ones), else 0; 0 for a free slot.  This is the
 * paper's mask: with a prefill it is l_am + l_q - 1 wide, l_am = L + 1.
 * mask: device uint8, >= batch rows of ld bytes.  Bytes at j >= L + T are
 * not touched.
 * Errors: EINVAL (null mask, ld < L + T), EHIP.
 */
baton_status baton_build_mask(const baton_cache* cache, uint8_t* mask, int64_t ld,
                              hipStream_t stream);

/* Bytes of device workspace baton_decode_attn needs for this cache in its
   current state.  Fixed while no prefill step has left holes; otherwise it
   grows with their number, so query it again after baton_step_advance and
   baton_kv_evict. */
size_t baton_decode_attn_workspace_bytes(const baton_cache* cache);

/*
 * Decode attention of one layer (sec. 2.1, "General architecture": dot products
 * of the query with the keys, scaling, softmax, weighted sum of the values).
 * For every live slot b and query head hq (kv-head h = hq / (n_q_heads /
 * n_kv_heads)): appends k_new[b][h], v_new[b][h] to the layer's cache as
 * column L, then
 *     out[b][hq] = softmax_j(scale * q[b][hq] . K[b][h][j]) . V[b][h][j]
 * over the slot's own columns j in [L - len_b, L] only; placeholder columns
 * are skipped, never read into arithmetic.  Free slots: nothing appended, out
 * rows set to 0.  Arithmetic in fp32; out rounded to nearest-even in the
 * cache's dtype.
 * Live rows' holes are skipped like placeholders.
 * q, out: device [batch][n_q_heads][head_dim]; k_new, v_new: device
 * [batch][n_kv_heads][head_dim]; all 16-byte aligned.
 * In a step registered by baton_shape_insert, q and out are
 * [batch][T][n_q_heads][head_dim] and k_new, v_new [batch][T][n_kv_heads]
 * [head_dim]: a live slot's position 0 is decoded as above (positions 1 .. T-1
 * are padding; only position 0 is appended); a slot being prefilled attends
 * causally over its own prompt -- its position T - l + i over prompt positions
 * T - l .. T - l + i -- and all l prompt positions are appended as columns
 * L + T - l .. L + T - 1.  out is written at positions that hold a token and at
 * position 0 of free slots (zeros); other positions are not touched.
 * scale = 0 selects
 * 1/sqrt(head_dim).  ws: device workspace of >= baton_decode_attn_workspace_bytes
 * bytes, 16-byte aligned, used by one cache at a time; its contents are the
 * library's between calls.  Call once per layer per step, then
 * baton_step_advance.
 * Errors: EINVAL (layer out of range, null pointer, ws too small, scale not
 * finite), ESTATE (layer already decoded this step), ECAPACITY (L + 1 >
 * capacity), EHIP.
 */
baton_status baton_decode_attn(baton_cache* cache, int32_t layer, const void* q, const void* k_new,
                               const void* v_new, void* out, float scale, void* ws, size_t ws_bytes,
                               hipStream_t stream);

/*
 * baton_decode_attn without a workspace, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  Same arguments, results and errors as
 * baton_decode_attn (bit for bit the same output), but the work list and the
 * split-K partial sums live in a scratch array of BATON_SCRATCH_BYTES that the
 * library keeps in the memory of each GPU it runs on until the process ends.
 * The call itself allocates nothing.  A step needs 32 bytes per work item, 16
 * per slot and 4 * (head_dim + 4) * n_q_heads bytes per work item of one
 * kv-head's items, each region rounded up to 256 bytes (work items: a
 * row's cached tokens plus one, cut every split tokens; about 550 items and
 * 18 MB for 128 slots of 8192 tokens with 64 query heads over 8 kv-heads).
 * Every call on one GPU shares that GPU's scratch and finds there what the
 * last call left: a step's first call (or the first after another cache used
 * the scratch) writes the work list again.  Calls whose work overlaps in time
 * on one GPU (on different streams) race on the scratch and give undefined
 * results; calls in one stream's order, for one cache or several, do not.
 * Errors: those of baton_decode_attn without the workspace's (EINVAL for a
 * null or misaligned pointer, a layer out of range or a scale not finite;
 * ESTATE; ECAPACITY), ESCRATCH (the step needs more than BATON_SCRATCH_BYTES:
 * nothing is enqueued; a larger split, baton_set_split_tokens, needs less),
 * EHIP (the GPU holding the cache or the scratch's address could not be
 * determined).
 */
#define BATON_SCRATCH_BYTES (64u << 20)
baton_status baton_decode_attn_noalloc(baton_cache* cache, int32_t layer, const void* q, const void* k_new,
                                       const void* v_new, void* out, float scale, hipStream_t stream);

/*
 * Enqueue the placeholder writes evictions still owe (see baton_kv_evict), so
 * that every non-live position holds the placeholder now.  Never needed for
 * correct results; for callers that read the ring directly.
 * Errors: EINVAL (null cache), EHIP.
 */
baton_status baton_cache_flush(baton_cache* cache, hipStream_t stream);

/*
 * Close the decode step once every layer has been decoded: L += 1 and every
 * live slot's length += 1 (sec. 4.1: cache and mask grow by one column per
 * iteration); after a prefill step L += T, every other live slot's length
 * += T (its new hole included) and the prefilled slots become live.  Host
 * metadata only.
 * Errors: ESTATE (some layer not decoded this step).
 */
baton_status baton_step_advance(baton_cache* cache);

/*
 * Current metadata: padded length L, ring base (physical column of logical
 * column 0), and per-slot lengths (host array of batch entries, 0 = free): a
 * live slot's span L - (column of its first token), holes included.  Any
 * output pointer may be NULL.
 */
baton_status baton_cache_query(const baton_cache* cache, int64_t* L, int64_t* base, int32_t* lens);

/*
 * Per-slot token counts (host array of batch entries, 0 = free): the span
 * without its holes, i.e. the length of the query's own history.  A caller
 * applying rotary position embeddings uses position tokens[b] for slot b's
 * next token.
 * Errors: EINVAL (null pointer).
 */
baton_status baton_cache_tokens(const baton_cache* cache, int32_t* tokens);

/*
 * Tuning: tokens per split of a row in baton_decode_attn, i.e. per work item
 * (one workgroup; a multiple of 64, 64 .. 4096), or 0 (the default) to let
 * each step choose from its total number of cached tokens (256 .. 4096, about
 * 4096 items per layer).  Changes
 * baton_decode_attn_workspace_bytes; only between steps.
 * Errors: EINVAL (out of range), ESTATE (inside a decode step).
 */
baton_status baton_set_split_tokens(baton_cache* cache, int32_t tokens);

/*
 * ---- A whole decode layer around the attention --------------------------
 * The paper serves llama2-7b (sec. 5; its layers as sec. 2.1 describes them:
 * W^Q, W^K, W^V projections, attention, feed-forward networks between).
 * These calls are the rest of such a layer, so that a decode step runs end to
 * end: RMS normalisation, the projections (the library's weight-streaming
 * kernel on packed weights, up to BATON_GEMM_MAX_ROWS rows), rotary position
 * embedding at each query's own position, the gated feed-forward, and fused
 * forms of the projections with the step that follows them.  bf16 only;
 * every output is rounded to nearest even.
 */
#define BATON_GEMM_MAX_ROWS 256

/*
 * y[r] (+)= x[r] . W^T for r < rows <= BATON_GEMM_MAX_ROWS (a linear layer at a
 * decode step's batch) on the library's weight-streaming kernel, which reads
 * the weight in a packed form made once per weight by baton_linear_pack.  The
 * weight dominates the traffic of such a product and is read about once from
 * HBM (rows past 64 are taken in chunks of 64 by workgroups dealt to the same
 * XCD one after the other, the later chunks finding the weight in that XCD's
 * L2); the packed form lets each wave stream it in contiguous 1 KB blocks.
 *
 * baton_linear_packed_bytes: bytes of the packed form of an [out_dim][in_dim]
 * weight: 2 * ceil(out_dim / 16) * 16 * ceil(in_dim / 32) * 32 (0 for sizes < 1).
 *
 * baton_linear_pack: writes the packed form of w (device [out_dim][in_dim],
 * bf16) into wp (device, caller-owned, baton_linear_packed_bytes, 16-byte
 * aligned): 16-row slices of w, each a run of 1 KB blocks, one per 32 columns,
 * block (s, t) holding at byte 16 l the eight elements
 * w[16 s + l % 16][32 t + 8 (l / 16) ...] (zeros past out_dim or in_dim).
 * Errors: EINVAL (null or misaligned pointer, sizes < 1 or not multiples of
 * 8), EDTYPE (not bf16), EHIP.
 *
 * baton_linear_packed: y[r] (+)= x[r] . W^T for r < rows <= BATON_GEMM_MAX_ROWS,
 * W given by its packed form wp; x device [rows][in_dim], y device
 * [rows][out_dim], both 16-byte aligned; accumulate = 1 adds to y (the
 * residual stream), 0 overwrites it.  fp32 accumulation;
 * when the output has few 16-row slices the sum is split along in_dim and the
 * fp32 partial sums, kept in ws (device, caller-owned; as many splits as
 * ws_bytes holds rows * out_dim floats for, none with ws_bytes = 0), are added
 * in a second launch in a fixed order.  Errors: EINVAL (null or misaligned
 * pointer, rows outside 1..BATON_GEMM_MAX_ROWS, sizes < 1 or not multiples of
 * 8, accumulate not 0/1), EDTYPE, EHIP.
 */
size_t baton_linear_packed_bytes(int32_t out_dim, int32_t in_dim);
baton_status baton_linear_pack(int32_t dtype, const void* w, void* wp, int32_t out_dim, int32_t in_dim,
                               hipStream_t stream);
baton_status baton_linear_packed(int32_t dtype, const void* x, const void* wp, void* y, int32_t rows,
                                 int32_t out_dim, int32_t in_dim, int32_t accumulate, void* ws, size_t ws_bytes,
                                 hipStream_t stream);

/*
 * baton_linear_packed, then the RMS norm of its output (the layer's residual
 * add followed by the next normalisation, as a llama2 decoder layer runs
 * them): y as baton_linear_packed leaves it, and y_norm (device
 * [rows][out_dim], 16-byte aligned, may alias y) = baton_rmsnorm(y, gain,
 * eps), bit for bit.  When the product splits along in_dim one kernel adds the
 * partial sums (and y with accumulate) and normalises each row, in place of
 * the addition's launch and the norm's launch.
 * Errors: those of baton_linear_packed and baton_rmsnorm (null or misaligned
 * gain / y_norm, eps < 0 or not finite: EINVAL).
 */
baton_status baton_linear_packed_rmsnorm(int32_t dtype, const void* x, const void* wp, void* y, int32_t rows,
                                         int32_t out_dim, int32_t in_dim, int32_t accumulate, const void* gain,
                                         float eps, void* y_norm, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * The gated feed-forward's first half in one call: y[r][j] = silu(g) * u with
 * g = x[r] . W[j], u = x[r] . W[F + j] (each rounded to bf16 as
 * baton_linear_packed would round them), silu(z) = z / (1 + e^-z), for
 * j < F = out_dim / 2 -- bit for bit baton_linear_packed with ws_bytes = 0
 * (the k-sum unsplit) into a [rows][out_dim] buffer followed by
 * baton_silu_mul, without writing or reading that buffer or a second launch.  W is [gate; up] ([out_dim][in_dim],
 * gate rows first) in its packed form wp; x device [rows <= BATON_GEMM_MAX_ROWS]
 * [in_dim], y device [rows][F].  Never splits along in_dim (no workspace).
 * Errors: EINVAL (null or misaligned pointer, rows outside
 * 1..BATON_GEMM_MAX_ROWS, out_dim not a positive multiple of 32, in_dim < 8 or
 * not a multiple of 8), EDTYPE, EHIP.
 */
baton_status baton_linear_packed_silu(int32_t dtype, const void* x, const void* wp, void* y, int32_t rows,
                                      int32_t out_dim, int32_t in_dim, hipStream_t stream);

/*
 * y[r] = x[r] / sqrt(mean_j x[r][j]^2 + eps) * gain: x, y device [rows][dim],
 * gain device [dim]; dim a multiple of 8.  y may alias x.
 * Errors: EINVAL (null or misaligned pointer, bad sizes, eps < 0), EDTYPE.
 */
baton_status baton_rmsnorm(int32_t dtype, const void* x, const void* gain, void* y, int32_t rows,
                           int32_t dim, float eps, hipStream_t stream);

/*
 * Split a fused projection qkv device [batch][(n_q_heads + 2 n_kv_heads)
 * head_dim] (query heads, then key heads, then value heads) into q
 * [batch][n_q_heads][head_dim], k_new and v_new [batch][n_kv_heads][head_dim],
 * rotating q and k: pair (i, i + head_dim/2) of a head by angle
 * pos_b * theta^(-2i/head_dim), pos_b = slot b's token count
 * (baton_cache_tokens), the position of the token being decoded.  The angles
 * are formed and reduced modulo 2 pi in double precision.  Decode steps only.
 * Errors: EINVAL (null pointer, theta <= 1), EDTYPE (cache not bf16), ESTATE
 * (a prefill is registered), EHIP.
 */
baton_status baton_rope_qkv(const baton_cache* cache, const void* qkv, void* q, void* k_new, void* v_new,
                            float theta, hipStream_t stream);

/*
 * out[r][j] = silu(gate_up[r][j]) * gate_up[r][dim + j], silu(z) = z / (1 + e^-z):
 * gate_up device [rows][2 dim] (gate, then up), out device [rows][dim].
 * Errors: EINVAL (null or misaligned pointer, dim not a multiple of 8), EDTYPE.
 */
baton_status baton_silu_mul(int32_t dtype, const void* gate_up, void* out, int32_t rows, int32_t dim,
                            hipStream_t stream);

/* Static English text of a status. */
const char* baton_status_string(baton_status status);

#ifdef __cplusplus
}
#endif

#endif /* BATON_H */
