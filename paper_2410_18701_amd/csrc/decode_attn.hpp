// Masked batched decode attention over the aligned ring cache, split over the
// sequence ("split-K") so that long and skewed rows spread over all CUs.
//
// Work item = (slot b, split c) x kv-head h: a range of at most S tokens t of
// row (layer, b, h) inside one run of consecutive tokens, where token t <
// len_b is cache column L - len_b + t and token len_b is the current token
// (k_new/v_new, appended to the cache by the wave that holds it).  Placeholder
// columns, holes included, are never addressed.  One workgroup of NW waves per
// item; wave w streams the w-th of NW equal contiguous shares of the item's
// tokens.  In a wave a token row of D elements is spread over LPT =
// D*elem/16 lanes (16 bytes each), so one wave instruction reads TPI = 64/LPT
// whole token rows; each of those TPI lane groups keeps its own online-softmax
// state (max m, sum l, weighted values acc) over the tokens it reads.  The
// lane groups merge by cross-lane moves, the waves through LDS.  An item that
// is its row's only one writes the output; otherwise it writes one (m, l, acc)
// partial record and combine_kernel merges the row's partials with the
// log-sum-exp rescale.  Rows up to S tokens (most rows at the usual S of a
// thousand tokens and more) thus need no partial record at all.  (Merging in
// the attention kernel by the last item to arrive would need an agent-scope
// release per item, which on gfx950 writes back the L2; measured, that costs
// far more than the second launch.)  A free slot gets one item that writes
// zeros.  Exponentials are base 2 with scale*log2(e) folded into q.
#pragma once

#include <type_traits>

#include "common.hpp"

#ifndef BATON_ATTN_NT
#define BATON_ATTN_NT 1      // non-temporal K/V loads (streamed once per layer and step)
#endif

namespace baton {

constexpr int kMetaThreads = 512;   // == BATON_MAX_BATCH

struct MetaArgs {
  int64_t L;
  int32_t batch;
  int32_t split;                    // tokens per item
  int32_t gather_max;               // tokens per gathered item; 0: no gathered items
  int32_t lens[kMetaThreads];       // cached tokens (span); 0 free; -1 prefilled this step (no item)
  uint8_t first[kMetaThreads];      // index of the row's first hole
  HoleList holes;
};

// One work item: the tokens [t_begin, t_end) of slot b's row (n = len_b
// cached tokens, -1 for a free slot), and where the row's items start and how
// many there are.  A gathered item (kGathered) instead lists its tokens: the
// token indices at [t_begin, t_end) of the workspace's gather list; with
// kCurrent it also takes the row's current token n.
struct Item {
  int4 span;     // (b, t_begin, t_end, n)
  int4 row;      // (first item of the row, items of the row, this item's index, flags)
};
constexpr int32_t kGathered = 1, kCurrent = 2;

// floor(x / d) for 0 <= x and 64 <= d (so that x * inv stays far inside
// int32): a float estimate from inv ~ 1/d, corrected to the exact quotient.
// The work list divides every run by the split; an integer division by a
// runtime value costs some 30 instructions.
__host__ __device__ __forceinline__ int32_t div_floor(int32_t x, int32_t d, float inv) {
  int32_t q = (int32_t)((float)x * inv);
  int32_t r = x - q * d;
  while (r < 0) {
    --q;
    r += d;
  }
  while (r >= d) {
    ++q;
    r -= d;
  }
  return q;
}

// The split and the reciprocals its divisions use.
struct Split {
  int32_t s;
  float inv, inv1;   // ~1 / s, ~1 / (s + 1)
};
__host__ __device__ __forceinline__ Split make_split(int32_t s) {
  return Split{s, 1.0f / (float)s, 1.0f / (float)(s + 1)};
}

// A row's share of the work list.  Each run of consecutive tokens is cut
// into pieces of at most `split` tokens -- unless gather_max > 0 and the run
// is shorter than gather_max: such short runs (what a row keeps between the
// holes of in-batch prefill steps, often a single token) are listed token by
// token and the list is cut into gathered items of at most gather_max tokens,
// so that a workgroup is not spent on each of them.  The current token of a
// short last run goes with the row's last gathered item, not into the list.
// short_piece(r) is called for each piece of r < split tokens.
struct RowPlan {
  int32_t items;       // work items of the row
  int32_t full;        // pieces of exactly `split` tokens
  int32_t listed;      // tokens in the gather list
  int32_t gathered;    // gathered items
  bool cur_gathered;   // the current token goes with the last gathered item
};

template <typename F>
__host__ __device__ __forceinline__ RowPlan row_plan(const HoleList& hl, int32_t first, int64_t L, int32_t n,
                                                     const Split& sp, int32_t gather_max, F&& short_piece) {
  RowPlan p{0, 0, 0, 0, false};
  if (n < 0) return p;
  if (n == 0) {
    p.items = 1;
    return p;
  }
  row_runs(hl, first, L, n, [&](int32_t t0, int32_t t1) {
    const int32_t len = t1 - t0;
    if (len < gather_max) {
      const bool last = t1 == n + 1;
      p.listed += len - (last ? 1 : 0);
      p.cur_gathered = p.cur_gathered || last;
    } else {
      const int32_t q = div_floor(len, sp.s, sp.inv), r = len - q * sp.s;
      p.full += q;
      p.items += q + (r > 0 ? 1 : 0);
      if (r > 0) short_piece(r);
    }
  });
  p.gathered = gather_max > 0 ? (p.listed + gather_max - 1) / gather_max : 0;
  if (p.cur_gathered && p.gathered == 0) p.gathered = 1;
  p.items += p.gathered;
  return p;
}

__host__ __device__ __forceinline__ RowPlan row_plan(const HoleList& hl, int32_t first, int64_t L, int32_t n,
                                                     int32_t split, int32_t gather_max) {
  return row_plan(hl, first, L, n, make_split(split), gather_max, [](int32_t) {});
}

// Size classes of the dispatch order: an item of t <= split tokens is in
// class t * kSizeClasses / (split + 1); the order runs from the largest class
// down.
constexpr int kSizeClasses = 64;

__device__ __forceinline__ int32_t size_class(int32_t t, const Split& sp) {
  return div_floor(t * kSizeClasses, sp.s + 1, sp.inv1);
}

// Class of a gathered item of t tokens (it may hold one more than `split`:
// a full list and the current token).
__device__ __forceinline__ int32_t gathered_class(int32_t t, const Split& sp) {
  return size_class(min(t, sp.s), sp);
}

// Sum of x over this lane and the lanes below it in the wave.
__device__ __forceinline__ int32_t wave_prefix_sum(int32_t x, int lane) {
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int32_t y = __shfl_up(x, off, kWave);
    if (lane >= off) x += y;
  }
  return x;
}

// Most tokens of a gathered item (the largest gather_max of the attention
// kernels: bf16 at head_dim 64).
constexpr int32_t kMaxGatherTokens = 128;

// Builds the per-step work list in the workspace: one descriptor per item,
// stored in the dispatch order -- the items from the most tokens to the fewest
// (a counting sort over size classes; the order within a class is arbitrary
// and affects no result) -- so that a workgroup needs a single load to start;
// the list of rows with several items (first item, item count, slot) for
// combine_kernel; and the gather list of the gathered items' tokens.  The
// items are those of row_plan.
// The attention workgroups are then dealt largest first, so that the ones that
// start last are short and the launch ends with little of the GPU idle.
// One thread per slot, and no row walks the hole list: the holes a row holds
// are the list from its first hole on (the host gives each row a first hole
// that ends after the row's first column), so the run after hole k -- from
// its end to the next hole's start, the last one to the current column L --
// is the same columns for every row that holds hole k.  The first wave plans
// these shared runs once (pieces, listed tokens, suffix sums over k, the
// listed columns of the short ones in LDS); a row's plan is then its own first
// run (to its first hole, or to its current token) plus the suffix sums at its
// first hole.  The full pieces (`split` tokens, all of the top class) take
// the first places of the list from one counter in LDS, one atomic per wave
// and loop trip (a full piece of every slot, then the next piece of every
// slot: workgroups that run at the same time read many rows -- measured faster
// than each slot's pieces side by side); the shorter pieces, the gathered
// items and a free slot's item take places through per-class counters after
// them.  Row offsets come from wave prefix sums, and a wave per row copies the
// row's listed tokens of the shared runs into its gather list.
__global__ void __launch_bounds__(kMetaThreads) meta_kernel(const MetaArgs a, Item* ws_items,
                                                            int4* ws_multi, int32_t* ws_gather) {
  static_assert(kSizeClasses == kWave, "one lane per size class");
  static_assert(kMaxHoles == kWave, "one lane per hole");
  constexpr int kWaves = kMetaThreads / kWave;
  __shared__ int32_t cursor[kSizeClasses];     // short items per class, then the class's next place
  __shared__ int32_t full_items, full_next, n_long, last_short;
  __shared__ int32_t wave_sum[3][kWaves];
  __shared__ int32_t first_col[kMaxHoles];        // start column of hole k (the end of a row's first run)
  __shared__ int32_t run_lo[kMaxHoles], run_hi[kMaxHoles];    // run k: columns [lo, hi)
  __shared__ int32_t long_run[kMaxHoles];         // the runs cut into pieces, in column order
  __shared__ int32_t suf_pieces[kMaxHoles + 1], suf_full[kMaxHoles + 1], suf_listed[kMaxHoles + 1];
  __shared__ int32_t sl_pos[kMaxHoles + 1];       // where run k's listed columns start in `sl`
  __shared__ int32_t holders[kMaxHoles + 1];      // live rows by first hole (run k's: those up to k)
  __shared__ int32_t sl[kMaxHoles * (kMaxGatherTokens - 1)];   // the short runs' listed columns
  __shared__ int32_t row_dst[kMetaThreads], row_c0[kMetaThreads], row_sl0[kMetaThreads],
      row_shared[kMetaThreads];
  const int b = threadIdx.x, lane = b % kWave, wv = b / kWave;
  const int32_t n = b < a.batch ? a.lens[b] : -1;
  const int32_t nh = a.holes.n;
  const int32_t fh = b < a.batch ? min((int32_t)a.first[b], nh) : nh;
  const int32_t gmax = a.gather_max;
  const int32_t L = (int32_t)a.L;   // logical columns fit int32 (the hole list holds them so)
  const Split sp = make_split(a.split);
  if (b < kSizeClasses) cursor[b] = 0;
  if (b <= kMaxHoles) holders[b] = 0;
  if (b == 0) full_items = full_next = 0;

  // The shared runs, planned by the first wave: lane k for hole k.
  if (wv == 0 && nh == 0) {   // none: every row's plan is its own single run
    suf_pieces[lane] = suf_full[lane] = suf_listed[lane] = sl_pos[lane] = 0;
    if (lane == 0) {
      suf_pieces[kMaxHoles] = suf_full[kMaxHoles] = suf_listed[kMaxHoles] = sl_pos[kMaxHoles] = 0;
      n_long = last_short = 0;
    }
  } else if (wv == 0) {
    const int k = lane;
    int32_t lo = 0, hi = 0, pieces = 0, full = 0, listed = 0;
    bool is_long = false;
    if (k < nh) {
      lo = a.holes.col[k][1];
      hi = k + 1 < nh ? a.holes.col[k + 1][0] : L + 1;
      const int32_t len = hi - lo;
      if (len < gmax) {
        listed = k == nh - 1 ? len - 1 : len;   // the last run holds the current token, never listed
      } else {
        full = div_floor(len, sp.s, sp.inv);
        pieces = full + (len - full * sp.s > 0 ? 1 : 0);
        is_long = true;
      }
      first_col[k] = a.holes.col[k][0];
    }
    run_lo[k] = lo;
    run_hi[k] = hi;
    // suffix sums over k: the total less the sum below k
    const int32_t p_pieces = wave_prefix_sum(pieces, lane), p_full = wave_prefix_sum(full, lane),
                  p_listed = wave_prefix_sum(listed, lane);
    const int32_t t_pieces = __shfl(p_pieces, kWave - 1, kWave), t_full = __shfl(p_full, kWave - 1, kWave),
                  t_listed = __shfl(p_listed, kWave - 1, kWave);
    suf_pieces[k] = t_pieces - (p_pieces - pieces);
    suf_full[k] = t_full - (p_full - full);
    suf_listed[k] = t_listed - (p_listed - listed);
    sl_pos[k] = p_listed - listed;
    const uint64_t longs = __ballot(is_long);
    if (is_long)
      long_run[__builtin_amdgcn_mbcnt_hi((uint32_t)(longs >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)longs, 0u))] = k;
    if (k == 0) {
      suf_pieces[kMaxHoles] = suf_full[kMaxHoles] = suf_listed[kMaxHoles] = 0;
      sl_pos[kMaxHoles] = t_listed;
      n_long = (int32_t)__popcll(longs);
      last_short = !((longs >> (nh - 1)) & 1u);
    }
  }
  __syncthreads();
  // The short runs' listed columns, a wave per run.
  for (int k = wv; k < nh; k += kWaves) {
    const int32_t at = sl_pos[k], cnt = sl_pos[k + 1] - at, lo = run_lo[k];
    for (int32_t i = lane; i < cnt; i += kWave) sl[at + i] = lo + i;
  }

  // This row's plan: its first run, then the shared runs from its first hole.
  int32_t items = 0, full = 0, listed = 0, first_listed = 0, gathered = 0;
  bool cur = false;
  const int32_t c0 = L - n;
  const int32_t f_end = fh < nh ? first_col[fh] - c0 : n + 1;   // the first run: tokens [0, f_end)
  if (n == 0) {
    items = 1;
    atomicAdd(&cursor[0], 1);
  } else if (n > 0) {
    if (f_end > 0) {
      if (f_end < gmax) {
        first_listed = fh < nh ? f_end : f_end - 1;
        cur = fh == nh;
      } else {
        const int32_t q = div_floor(f_end, sp.s, sp.inv), r = f_end - q * sp.s;
        full = q;
        items = q + (r > 0 ? 1 : 0);
        if (r > 0) atomicAdd(&cursor[size_class(r, sp)], 1);
      }
    }
    if (fh < nh) cur = last_short != 0;
    listed = first_listed + suf_listed[fh];
    full += suf_full[fh];
    items += suf_pieces[fh];
    gathered = gmax > 0 ? (listed + gmax - 1) / gmax : 0;
    if (cur && gathered == 0) gathered = 1;
    items += gathered;
    if (fh < nh) atomicAdd(&holders[fh], 1);   // a row past the last hole holds no shared run
    for (int32_t j = 0; j < gathered; ++j) {
      const int32_t t = min(gmax, listed - j * gmax) + (cur && j == gathered - 1 ? 1 : 0);
      atomicAdd(&cursor[gathered_class(t, sp)], 1);
    }
    atomicAdd(&full_items, full);
  }
  const int32_t multi = items > 1 ? 1 : 0;
  int32_t s_cnt = wave_prefix_sum(items, lane);
  int32_t s_multi = wave_prefix_sum(multi, lane);
  int32_t s_list = wave_prefix_sum(listed, lane);
  if (lane == kWave - 1) {
    wave_sum[0][wv] = s_cnt;
    wave_sum[1][wv] = s_multi;
    wave_sum[2][wv] = s_list;
  }
  __syncthreads();   // wave totals, row counts by first hole and the class counts complete
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const int32_t c0w = wave_sum[0][w], c1 = wave_sum[1][w], c2 = wave_sum[2][w];
    if (w < wv) {
      s_cnt += c0w;
      s_multi += c1;
      s_list += c2;
    }
  }
  const int32_t first = s_cnt - items;     // the row's first item: its partial records start here
  const int32_t list0 = s_list - listed;   // the row's tokens in the gather list start here
  const bool any_shared = sl_pos[kMaxHoles] > 0;   // listed tokens in the shared runs
  if (any_shared) {
    row_dst[b] = list0 + first_listed;       // and those of its shared runs here
    row_c0[b] = c0;
    row_sl0[b] = sl_pos[fh];
    row_shared[b] = n > 0 ? suf_listed[fh] : 0;
  }
  if (wv == 0) {
    // The shorter pieces of the long shared runs: one per row that holds the
    // run.  Then the start of each class's places: after every full piece and
    // every larger class (no other item is in a class above the full pieces').
    if (nh > 0) {
      const int32_t hold = wave_prefix_sum(holders[lane], lane);   // rows whose first hole is <= lane
      if (lane < nh) {
        const int32_t len = run_hi[lane] - run_lo[lane];
        if (len >= gmax) {
          const int32_t r = len - div_floor(len, sp.s, sp.inv) * sp.s;
          if (r > 0 && hold > 0) atomicAdd(&cursor[size_class(r, sp)], hold);
        }
      }
      __threadfence_block();   // the wave's adds land before its lanes read the counts
    }
    const int k = kSizeClasses - 1 - lane;
    const int32_t c = cursor[k];
    cursor[k] = full_items + wave_prefix_sum(c, lane) - c;
  }
  __syncthreads();
  // The descriptors, each at its place in the dispatch order; an item's own
  // index (its row's first item + its rank in the row) numbers its partial
  // record.
  if (n == 0) {
    ws_items[atomicAdd(&cursor[0], 1)] = Item{make_int4(b, 0, 0, -1), make_int4(first, 1, first, 0)};
  } else if (n > 0) {
    int32_t c = first;
    auto pieces_of = [&](int32_t t0, int32_t t1) {   // a long run, cut at every `split` tokens
      for (int32_t t = t0; t < t1; t += sp.s, ++c) {
        const int32_t te = min(t + sp.s, t1);
        int32_t pos;
        if (te - t == sp.s) {
          // the wave's lanes with a full piece take consecutive places, in lane order
          const uint64_t act = __ballot(1);
          const int32_t rank =
              (int32_t)__builtin_amdgcn_mbcnt_hi((uint32_t)(act >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)act, 0u));
          int32_t at = 0;
          if (rank == 0) at = atomicAdd(&full_next, (int32_t)__popcll(act));
          pos = __builtin_amdgcn_readfirstlane(at) + rank;
        } else {
          pos = atomicAdd(&cursor[size_class(te - t, sp)], 1);
        }
        ws_items[pos] = Item{make_int4(b, t, te, n), make_int4(first, items, c, 0)};
      }
    };
    if (f_end > 0) {
      if (f_end < gmax) {
        for (int32_t t = 0; t < first_listed; ++t) ws_gather[list0 + t] = t;
      } else {
        pieces_of(0, f_end);
      }
    }
    const int32_t nl = n_long;
    for (int32_t i = 0; i < nl; ++i) {
      const int32_t k = long_run[i];
      if (k >= fh) pieces_of(run_lo[k] - c0, run_hi[k] - c0);
    }
    for (int32_t j = 0; j < gathered; ++j, ++c) {
      const int32_t g0 = list0 + j * gmax, g1 = min(g0 + gmax, list0 + listed);
      const int32_t flags = kGathered | (cur && j == gathered - 1 ? kCurrent : 0);
      const int32_t t = min(gmax, listed - j * gmax) + (cur && j == gathered - 1 ? 1 : 0);
      const int32_t pos = atomicAdd(&cursor[gathered_class(t, sp)], 1);
      ws_items[pos] = Item{make_int4(b, g0, g1, n), make_int4(first, items, c, flags)};
    }
  }
  if (multi) ws_multi[s_multi - 1] = make_int4(first, items, b, 0);
  // Every row's listed tokens of the shared runs, a wave per row: wave w
  // takes rows w, w + kWaves, ..., read one per lane, and copies those with any.
  static_assert(kWaves * kWave == kMetaThreads, "a lane per row");
  if (!any_shared) return;
  const int r = wv + kWaves * lane;
  const int32_t cnt = r < a.batch ? row_shared[r] : 0;
  const int32_t dst = row_dst[r], src = row_sl0[r], rc0 = row_c0[r];
  for (uint64_t m = __ballot(cnt > 0); m != 0; m &= m - 1) {
    const int j = (int)__builtin_ctzll(m);
    const int32_t cj = __shfl(cnt, j, kWave), dj = __shfl(dst, j, kWave), sj = __shfl(src, j, kWave),
                  oj = __shfl(rc0, j, kWave);
    for (int32_t i = lane; i < cj; i += kWave) ws_gather[dj + i] = sl[sj + i] - oj;
  }
}

struct AttnArgs {
  const uint32_t* k;         // the layer's ring rows [batch][n_kv_heads][cap][D], 32-bit words
  uint32_t* v;
  uint32_t* k_w;             // same as k, writable (append)
  const uint32_t* q;         // [batch][tw][n_q_heads][D], position 0 decoded
  const uint32_t* knew;      // [batch][tw][n_kv_heads][D]
  const uint32_t* vnew;
  uint32_t* out;             // [batch][tw][n_q_heads][D]
  const Item* items;         // workspace: the work list in dispatch order
  const int4* multi;         // rows with several items: (first item, count, slot)
  const int32_t* gather;     // tokens of the gathered items
  float* partial;            // [n_kv_heads][n_items][G][D + 4]
  int64_t cap, base, L;
  int32_t batch, n_kv_heads, split, n_items;
  int32_t tw;                // input positions per row (1; T in a prefill step)
  float qscale;              // scale * log2(e)
};

template <typename T, int D>
struct Geometry {
  static constexpr int kEpl = Lane16<T>::kElems;   // elements per lane
  static constexpr int kLpt = D / kEpl;            // lanes per token row
  static constexpr int kTpi = kWave / kLpt;        // token rows per wave instruction
  static constexpr int kVpt = kLpt;                // 16-byte vectors per token row
  static_assert(kLpt >= 4 && kLpt <= 32, "token row must span 4..32 lanes");
};

// Word 3 of a raw buffer resource on gfx9-family GPUs (no format conversion).
constexpr int32_t kBufferWord3 = 0x00020000;

__device__ __forceinline__ u32x4 load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  // aux bit 1: non-temporal (streamed once per layer and step)
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, BATON_ATTN_NT ? 2 : 0));
}

// Online-softmax update of one lane group with U token rows per lane group:
// scores by a dot product over the group's lanes (DPP), running max m, sum l
// and value accumulator acc rescaled by exp2(m_old - m_new).
template <typename T, int G, int U, int EPL, int LPT>
__device__ __forceinline__ void online_update(const u32x4 (&kw)[U], const u32x4 (&vw)[U],
                                              const bool (&valid)[U], const float (&qf)[G][EPL],
                                              float (&m)[G], float (&l)[G], float (&acc)[G][EPL]) {
  float s[U][G];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    float kf[EPL];
    Lane16<T>::widen(kw[u], kf);
#pragma unroll
    for (int gi = 0; gi < G; ++gi) {
      float d = 0.f;
#pragma unroll
      for (int e = 0; e < EPL; ++e) d = fmaf(qf[gi][e], kf[e], d);
      d = group_sum<LPT>(d);
      s[u][gi] = valid[u] ? d : -INFINITY;
    }
  }
#pragma unroll
  for (int gi = 0; gi < G; ++gi) {
    float mt = m[gi];
#pragma unroll
    for (int u = 0; u < U; ++u) mt = fmaxf(mt, s[u][gi]);
    const float ref = mt == -INFINITY ? 0.f : mt;
    const float alpha = fast_exp2(m[gi] - ref);
    l[gi] *= alpha;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[gi][e] *= alpha;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float p = fast_exp2(s[u][gi] - ref);
      l[gi] += p;
      float vf[EPL];
      Lane16<T>::widen(vw[u], vf);
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[gi][e] = fmaf(p, vf[e], acc[gi][e]);
    }
    m[gi] = mt;
  }
}

// Log-sum-exp merge of a row's partial records (m, l, acc[D]) for one query
// head.  Up to eight records (most rows): every lane loads all of them at
// once (two, four or eight records' worth) -- each record's m and l, and its
// own D/64 elements -- and merges them in record order after that one round
// trip.  More: lane i reads record i's m
// (64 at a time) and the wave reduces the max; then every lane accumulates its
// elements over the records, eight records' loads in flight at a time, with
// the weights broadcast from the lanes that computed them.
template <typename T, int D, int G>
__device__ __forceinline__ void merge_row(const float* base, int32_t count, uint32_t* outw,
                                          int lane) {
  constexpr int REC = D + 4;
  constexpr int PER = D / kWave;   // elements per lane (1 or 2)
  constexpr int64_t STRIDE = (int64_t)G * REC;
  auto store = [&](const float (&o)[PER], float inv) {
    if constexpr (T::kBytes == 4) {
#pragma unroll
      for (int e = 0; e < PER; ++e) outw[lane * PER + e] = __float_as_uint(o[e] * inv);
    } else {
      uint16_t* out16 = reinterpret_cast<uint16_t*>(outw);
#pragma unroll
      for (int e = 0; e < PER; ++e) out16[lane * PER + e] = (uint16_t)f32_to_bf16_rne(o[e] * inv);
    }
  };
  // count <= N records, all loaded at once (past the last: the last again, weighted 0)
  auto few = [&](auto n_tag) {
    constexpr int N = decltype(n_tag)::value;
    float mv[N], lv[N], v[N][PER];
#pragma unroll
    for (int j = 0; j < N; ++j) {
      const float* rec = base + (int64_t)min(j, count - 1) * STRIDE;
      mv[j] = rec[D];
      lv[j] = rec[D + 1];
#pragma unroll
      for (int e = 0; e < PER; ++e) v[j][e] = rec[lane * PER + e];
    }
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < N; ++j) mx = j < count ? fmaxf(mx, mv[j]) : mx;
    float l = 0.f, o[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) o[e] = 0.f;
#pragma unroll
    for (int j = 0; j < N; ++j) {
      const float w = j < count && mv[j] != -INFINITY ? exp2f(mv[j] - mx) : 0.f;
      l += w * lv[j];
#pragma unroll
      for (int e = 0; e < PER; ++e) o[e] = fmaf(w, v[j][e], o[e]);
    }
    store(o, 1.f / l);
  };
  if (count <= 2) return few(std::integral_constant<int, 2>{});
  if (count <= 4) return few(std::integral_constant<int, 4>{});
  if (count <= 8) return few(std::integral_constant<int, 8>{});
  float mm = -INFINITY;
  for (int32_t i0 = 0; i0 < count; i0 += kWave) {
    const int32_t i = i0 + lane;
    mm = fmaxf(mm, i < count ? base[i * STRIDE + D] : -INFINITY);
  }
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) mm = fmaxf(mm, __shfl_xor(mm, off, kWave));
  float l = 0.f, o[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) o[e] = 0.f;
  for (int32_t i0 = 0; i0 < count; i0 += kWave) {
    const int32_t i = i0 + lane;
    float w = 0.f;
    if (i < count) {
      const float mi = base[i * STRIDE + D];
      w = mi == -INFINITY ? 0.f : exp2f(mi - mm);
      l += w * base[i * STRIDE + D + 1];
    }
    const int32_t nrec = min(kWave, count - i0);
    for (int32_t j0 = 0; j0 < nrec; j0 += 8) {
      float v[8][PER];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float* rec = base + (int64_t)(i0 + min(j0 + j, nrec - 1)) * STRIDE;
#pragma unroll
        for (int e = 0; e < PER; ++e) v[j][e] = rec[lane * PER + e];
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float wj = j0 + j < nrec ? __shfl(w, j0 + j, kWave) : 0.f;
#pragma unroll
        for (int e = 0; e < PER; ++e) o[e] = fmaf(wj, v[j][e], o[e]);
      }
    }
  }
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) l += __shfl_xor(l, off, kWave);
  store(o, 1.f / l);
}

#ifndef BATON_ATTN_WAVES_PER_EU
#define BATON_ATTN_WAVES_PER_EU 2   // keeps the register budget at two waves per SIMD (0: compiler's choice)
#endif

// The work unit (item, kv-head) of this workgroup: workgroups are dealt in
// the work list's dispatch order (largest items first), all kv-heads of an
// item next to each other; one load gives the item's descriptor.
__device__ __forceinline__ Item work_unit(const AttnArgs& a, int32_t& item, int32_t& h) {
  const int32_t k = blockIdx.x;
  const Item d = a.items[k / a.n_kv_heads];
  item = d.row.z;
  h = k % a.n_kv_heads;
  return d;
}

// Merge of the NW waves of a workgroup, each holding the online-softmax state
// of its share of the item's tokens for the G query heads: wave w has put its
// max, sum and accumulator into sm_m[w][gi], sm_l[w][gi] and the G x D floats
// at sm_acc + w * acc_stride ([gi][d]; a wave with no tokens: max -inf, sum
// 0).  Every thread of the workgroup
// then merges pairs of output elements with the log-sum-exp rescale and writes
// the item's output (the item is its row's only one) or its partial record.
template <typename T, int D, int G, int NW>
__device__ __forceinline__ void wg_merge_write(const float (&sm_m)[NW][G], const float (&sm_l)[NW][G],
                                               const float* sm_acc, int acc_stride, bool whole_row,
                                               uint32_t* outw, float* rec0, int tid) {
  constexpr int REC = D + 4;
  for (int p = tid; p < G * D / 2; p += NW * kWave) {
    const int gi = p / (D / 2), e = 2 * (p % (D / 2));
    float mm = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) mm = fmaxf(mm, sm_m[w][gi]);
    float l = 0.f, o0 = 0.f, o1 = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float mw = sm_m[w][gi];
      const float f = mw == -INFINITY ? 0.f : exp2f(mw - mm);
      l = fmaf(f, sm_l[w][gi], l);
      o0 = fmaf(f, sm_acc[w * acc_stride + gi * D + e], o0);
      o1 = fmaf(f, sm_acc[w * acc_stride + gi * D + e + 1], o1);
    }
    if (whole_row) {
      const float inv = 1.f / l;
      if constexpr (T::kBytes == 4) {
        outw[gi * D + e] = __float_as_uint(o0 * inv);
        outw[gi * D + e + 1] = __float_as_uint(o1 * inv);
      } else {
        outw[(gi * D + e) / 2] = f32_to_bf16_rne(o0 * inv) | (f32_to_bf16_rne(o1 * inv) << 16);
      }
    } else {
      float* rec = rec0 + gi * REC;
      rec[e] = o0;
      rec[e + 1] = o1;
      if (e == 0) {
        rec[D] = mm;
        rec[D + 1] = l;
      }
    }
  }
}

// Tokens [wb, we) of an item [t_begin, t_end) that wave w of NW streams: equal
// contiguous shares, whole loop steps of STEP tokens except at the end.
template <int NW, int STEP>
__device__ __forceinline__ void wave_share(int32_t t_begin, int32_t t_end, int w, int32_t& wb,
                                           int32_t& we) {
  const int32_t per = (t_end - t_begin + NW - 1) / NW;
  const int32_t part = (per + STEP - 1) / STEP * STEP;
  wb = min(t_begin + w * part, t_end);
  we = min(wb + part, t_end);
}

template <typename T, int D, int G, int U, int NW>
__global__ void __launch_bounds__(kWave * NW)
#if BATON_ATTN_WAVES_PER_EU > 0
__attribute__((amdgpu_waves_per_eu(BATON_ATTN_WAVES_PER_EU)))
#endif
attn_kernel(const AttnArgs a) {
  using Geo = Geometry<T, D>;
  constexpr int EPL = Geo::kEpl, LPT = Geo::kLpt, TPI = Geo::kTpi, VPT = Geo::kVpt;
  constexpr int REC = D + 4;   // floats per partial record
  __shared__ float sm_m[NW][G], sm_l[NW][G];
  __shared__ float sm_acc[NW][G][D];
  int32_t item, h;
  const Item desc = work_unit(a, item, h);
  const int tid = threadIdx.x;
  // wave of the workgroup, as a scalar: the loop bounds derived from it are uniform
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int lane = tid % kWave;
  const int r = lane / LPT;        // token row within an instruction
  const int cl = lane % LPT;       // 16-byte slice of the row

  const int4 it = desc.span;
  const int4 rw = desc.row;
  const int b = it.x;
  const int32_t n = it.w;          // cached tokens; token n is the current one
  const int64_t bt = (int64_t)b * a.tw;   // input row of the slot's position 0
  uint32_t* outw = a.out + ((bt * a.n_kv_heads + h) * G) * (D * T::kBytes / 4);
  if (n < 0) {                     // free slot: the output rows are zero
    for (int v = tid; v < G * VPT; v += NW * kWave) reinterpret_cast<u32x4*>(outw)[v] = u32x4{0, 0, 0, 0};
    return;
  }
  const bool whole_row = rw.y == 1;
  constexpr int32_t STEP = TPI * U;
  int32_t t_begin, t_end;          // this wave's share of the item's tokens
  wave_share<NW, STEP>(it.y, it.z, w, t_begin, t_end);

  const int64_t row = (int64_t)b * a.n_kv_heads + h;   // within the layer's rows
  constexpr uint32_t ROWB = VPT * 16;                     // bytes per token row
  const uint32_t ring_bytes = (uint32_t)a.cap * ROWB;
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(a.k) + row * a.cap * VPT * 4, 0,
                                        ring_bytes, kBufferWord3);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc(a.v + row * a.cap * VPT * 4, 0, ring_bytes, kBufferWord3);
  const uint32_t start = (uint32_t)ring_add(a.base, a.L - n, a.cap);   // ring column of token 0
  const uint32_t cap = (uint32_t)a.cap;
  const u32x4* knew = reinterpret_cast<const u32x4*>(a.knew) + (bt * a.n_kv_heads + h) * VPT;
  const u32x4* vnew = reinterpret_cast<const u32x4*>(a.vnew) + (bt * a.n_kv_heads + h) * VPT;

  // Query slices of the G heads that share kv-head h, pre-scaled.
  float qf[G][EPL];
#pragma unroll
  for (int gi = 0; gi < G; ++gi) {
    const u32x4 qw = reinterpret_cast<const u32x4*>(a.q)[((bt * a.n_kv_heads + h) * G + gi) * VPT + cl];
    Lane16<T>::widen(qw, qf[gi]);
#pragma unroll
    for (int e = 0; e < EPL; ++e) qf[gi][e] *= a.qscale;
  }

  float m[G], l[G], acc[G][EPL];
#pragma unroll
  for (int gi = 0; gi < G; ++gi) {
    m[gi] = -INFINITY;
    l[gi] = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[gi][e] = 0.f;
  }

  // Cached tokens of the share, software-pipelined: the 2U loads of the next
  // iteration are in flight while the current one is computed.  A token past
  // the end gets an offset beyond the buffer's range, which the hardware
  // answers with zeros and no memory access (its score is then set to -inf).
  // The loads are issued unconditionally, also past the end: a load under a
  // branch would make the wait before the computation wait for it too.
  const int32_t c_end = min(t_end, n);
  auto issue = [&](int32_t tt, u32x4 (&kw)[U], u32x4 (&vw)[U], bool (&valid)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int32_t t = tt + u * TPI + r;
      valid[u] = t < c_end;
      uint32_t col = start + (uint32_t)t;
      col = col >= cap ? col - cap : col;
      const uint32_t off = valid[u] ? col * ROWB + cl * 16u : 0x80000000u;
      kw[u] = load16(rk, off);
      vw[u] = load16(rv, off);
    }
  };
  const bool gathered = (rw.w & kGathered) != 0;
  if (gathered) {
    // A gathered item: its share of the listed tokens (short runs of a
    // holey row), usually a single pass; the token index first, then the rows.
    for (int32_t i0 = t_begin; i0 < t_end; i0 += STEP) {
      int32_t tok[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int32_t i = i0 + u * TPI + r;
        tok[u] = i < t_end ? a.gather[i] : -1;
      }
      u32x4 kw[U], vw[U];
      bool valid[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        valid[u] = tok[u] >= 0;
        uint32_t col = start + (uint32_t)max(tok[u], 0);
        col = col >= cap ? col - cap : col;
        const uint32_t off = valid[u] ? col * ROWB + cl * 16u : 0x80000000u;
        kw[u] = load16(rk, off);
        vw[u] = load16(rv, off);
      }
      online_update<T, G, U, EPL, LPT>(kw, vw, valid, qf, m, l, acc);
    }
  } else if (t_begin < c_end) {
    u32x4 ka[U], va[U], kb[U], vb[U];
    bool la[U], lb[U];
    const int32_t n_iter = (c_end - t_begin + STEP - 1) / STEP;
    issue(t_begin, ka, va, la);
    int32_t tt = t_begin;
    for (int32_t i = 0; i + 2 <= n_iter; i += 2) {
      issue(tt + STEP, kb, vb, lb);
      __builtin_amdgcn_sched_barrier(0);   // keep the loads ahead of the computation
      online_update<T, G, U, EPL, LPT>(ka, va, la, qf, m, l, acc);
      issue(tt + 2 * STEP, ka, va, la);
      __builtin_amdgcn_sched_barrier(0);
      online_update<T, G, U, EPL, LPT>(kb, vb, lb, qf, m, l, acc);
      tt += 2 * STEP;
    }
    if (n_iter & 1) online_update<T, G, U, EPL, LPT>(ka, va, la, qf, m, l, acc);
  }

  // The current token: read from k_new / v_new by lane group 0, appended to
  // the cache as column L by the wave that holds it (once per row; of a
  // gathered item, by its first wave).
  if (gathered ? (rw.w & kCurrent) != 0 && w == 0 : n >= t_begin && n < t_end) {
    u32x4 kw[1] = {knew[cl]}, vw[1] = {vnew[cl]};
    bool valid[1] = {r == 0};
    online_update<T, G, 1, EPL, LPT>(kw, vw, valid, qf, m, l, acc);
    if (r == 0) {
      const uint32_t col = (uint32_t)ring_add(start, n, a.cap);
      reinterpret_cast<u32x4*>(a.k_w)[row * a.cap * VPT + (int64_t)col * VPT + cl] = kw[0];
      reinterpret_cast<u32x4*>(a.v)[row * a.cap * VPT + (int64_t)col * VPT + cl] = vw[0];
    }
  }

  // Merge the TPI lane groups of the wave.
#pragma unroll
  for (int off = LPT; off < kWave; off <<= 1) {
#pragma unroll
    for (int gi = 0; gi < G; ++gi) {
      const float mo = __shfl_xor(m[gi], off, kWave);
      const float lo = __shfl_xor(l[gi], off, kWave);
      const float mm = fmaxf(m[gi], mo);
      const float fa = m[gi] == -INFINITY ? 0.f : exp2f(m[gi] - mm);
      const float fb = mo == -INFINITY ? 0.f : exp2f(mo - mm);
      l[gi] = l[gi] * fa + lo * fb;
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        const float ao = __shfl_xor(acc[gi][e], off, kWave);
        acc[gi][e] = acc[gi][e] * fa + ao * fb;
      }
      m[gi] = mm;
    }
  }

  // Merge the waves through LDS and write the output or the partial record.
  if (r == 0) {
#pragma unroll
    for (int gi = 0; gi < G; ++gi) {
#pragma unroll
      for (int e = 0; e < EPL; ++e) sm_acc[w][gi][cl * EPL + e] = acc[gi][e];
      if (cl == 0) {
        sm_m[w][gi] = m[gi];
        sm_l[w][gi] = l[gi];
      }
    }
  }
  __syncthreads();
  float* rec0 = a.partial + (((int64_t)h * a.n_items + item) * G) * REC;
  wg_merge_write<T, D, G, NW>(sm_m, sm_l, &sm_acc[0][0][0], G * D, whole_row, outw, rec0, tid);
}

// One wave per (row with several items, query head): the log-sum-exp merge
// of the row's partials.
template <typename T, int D, int G>
__global__ void __launch_bounds__(kWave) combine_kernel(const AttnArgs a) {
  constexpr int REC = D + 4;
  const int4 mr = a.multi[blockIdx.x];
  const int hq = blockIdx.y, h = hq / G, gi = hq % G;
  uint32_t* outw = a.out + ((int64_t)mr.z * a.tw * a.n_kv_heads * G + hq) * (D * T::kBytes / 4);
  const float* base = a.partial + (((int64_t)h * a.n_items + mr.x) * G + gi) * REC;
  merge_row<T, D, G>(base, mr.y, outw, threadIdx.x);
}

}  // namespace baton
