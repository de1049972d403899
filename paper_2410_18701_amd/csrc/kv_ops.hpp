// KV-cache shaping kernels: placeholder fill, end-aligned embed / evict scrub /
// extract, attention-mask build.  Pure data movement: every kernel streams 16-byte
// vectors per lane with non-temporal stores (the data is not re-read before it
// leaves the caches).
#pragma once

#include "common.hpp"

namespace baton {

constexpr int kMaxSegs = 32;   // inserts (or evictions) per launch
constexpr int kCopyThreads = 256;
constexpr int kCopyVecs = 4;   // 16-byte vectors per thread per tile

// Work of one launch: up to kMaxSegs row sets.  Segment i covers, in every
// layer and kv-head and for both K and V, `len[i]` tokens of slot `slot[i]`
// starting at physical ring column `col0[i]`.  The contiguous side ext[i] is
// [layer][head][ext_len[i]][D] and the segment maps to its tokens
// ext_t0[i] .. ext_t0[i] + len[i] - 1.  With `extract` clear, the segment is
// copied from ext[i] into the ring, or the placeholder is written when ext[i]
// is null; with `extract` set the ring columns are copied out into ext[i].
struct SegArgs {
  uint32_t* k;              // ring buffers, viewed as 32-bit words
  uint32_t* v;
  int64_t cap;              // ring columns
  int64_t layer_vec;        // 16-byte vectors from one layer's rows to the next layer's
  int32_t n_layers, batch, n_kv_heads;
  int32_t n_segs;
  int32_t extract;          // 1: ring -> ext, 0: ext (or placeholder) -> ring, 2: ring row -> ring row
  uint32_t fill_word;       // placeholder bits replicated to a 32-bit word
  int32_t slot[kMaxSegs];
  int32_t len[kMaxSegs];
  int32_t tiles_per_row[kMaxSegs];
  int64_t col0[kMaxSegs];
  int64_t tile_end[kMaxSegs];           // inclusive prefix of tiles over segments
  int32_t dst_slot[kMaxSegs];           // mode 2: the slot whose row receives the columns
  int32_t ext_len[kMaxSegs];            // tokens per (layer, head) of the contiguous side
  int32_t ext_t0[kMaxSegs];             // its first token of this segment
  uint32_t* kext[kMaxSegs];             // contiguous side; null: placeholders
  uint32_t* vext[kMaxSegs];
};

// VPT = 16-byte vectors per token row (head_dim * elem_bytes / 16).  One block
// moves one tile of TT = kCopyThreads * kCopyVecs / VPT tokens of one row.
template <int VPT>
__global__ void __launch_bounds__(kCopyThreads) seg_kernel(const SegArgs a) {
  constexpr int TT = kCopyThreads * kCopyVecs / VPT;
  const int64_t g = blockIdx.x;
  int i = 0;
  while (i < a.n_segs - 1 && g >= a.tile_end[i]) ++i;
  const int64_t local = g - (i > 0 ? a.tile_end[i - 1] : 0);
  const int32_t tpr = a.tiles_per_row[i];
  const int64_t row = local / tpr;
  const int32_t tile = (int32_t)(local - row * tpr);
  const int32_t lh_count = a.n_layers * a.n_kv_heads;
  const int32_t which = (int32_t)(row / lh_count);          // 0: K, 1: V
  const int32_t lh = (int32_t)(row - (int64_t)which * lh_count);
  const int32_t layer = lh / a.n_kv_heads, h = lh - layer * a.n_kv_heads;
  const int32_t len = a.len[i];
  const int32_t t0 = tile * TT;
  const int32_t nt = min(TT, len - t0);

  u32x4* ring = reinterpret_cast<u32x4*>(which ? a.v : a.k) + layer * a.layer_vec +
               ((int64_t)a.slot[i] * a.n_kv_heads + h) * a.cap * VPT;
  u32x4* ext = reinterpret_cast<u32x4*>(which ? a.vext[i] : a.kext[i]);
  if (ext) ext += (((int64_t)layer * a.n_kv_heads + h) * a.ext_len[i] + a.ext_t0[i] + t0) * VPT;
  const int64_t c0 = ring_add(a.col0[i], t0, a.cap);

  u32x4 val[kCopyVecs];
  const u32x4 fill = {a.fill_word, a.fill_word, a.fill_word, a.fill_word};
  if (a.extract == 2) {     // the same ring columns of another slot's row
    u32x4* dst = reinterpret_cast<u32x4*>(which ? a.v : a.k) + layer * a.layer_vec +
                 ((int64_t)a.dst_slot[i] * a.n_kv_heads + h) * a.cap * VPT;
#pragma unroll
    for (int r = 0; r < kCopyVecs; ++r) {
      const int idx = threadIdx.x + r * kCopyThreads;
      if (idx < nt * VPT) {
        const int t = idx / VPT, e = idx - (idx / VPT) * VPT;
        val[r] = __builtin_nontemporal_load(ring + ring_add(c0, t, a.cap) * VPT + e);
      }
    }
#pragma unroll
    for (int r = 0; r < kCopyVecs; ++r) {
      const int idx = threadIdx.x + r * kCopyThreads;
      if (idx < nt * VPT) {
        const int t = idx / VPT, e = idx - (idx / VPT) * VPT;
        __builtin_nontemporal_store(val[r], dst + ring_add(c0, t, a.cap) * VPT + e);
      }
    }
    return;
  }
  if (a.extract) {
#pragma unroll
    for (int r = 0; r < kCopyVecs; ++r) {
      const int idx = threadIdx.x + r * kCopyThreads;
      if (idx < nt * VPT) {
        const int t = idx / VPT, e = idx - (idx / VPT) * VPT;
        val[r] = __builtin_nontemporal_load(ring + ring_add(c0, t, a.cap) * VPT + e);
      }
    }
#pragma unroll
    for (int r = 0; r < kCopyVecs; ++r) {
      const int idx = threadIdx.x + r * kCopyThreads;
      if (idx < nt * VPT) __builtin_nontemporal_store(val[r], ext + idx);
    }
    return;
  }
#pragma unroll
  for (int r = 0; r < kCopyVecs; ++r) {
    const int idx = threadIdx.x + r * kCopyThreads;
    val[r] = fill;
    if (ext && idx < nt * VPT) val[r] = __builtin_nontemporal_load(ext + idx);
  }
#pragma unroll
  for (int r = 0; r < kCopyVecs; ++r) {
    const int idx = threadIdx.x + r * kCopyThreads;
    if (idx < nt * VPT) {
      const int t = idx / VPT, e = idx - (idx / VPT) * VPT;
      const int64_t col = ring_add(c0, t, a.cap);
      __builtin_nontemporal_store(val[r], ring + col * VPT + e);
    }
  }
}

// Writes the placeholder over the n_vec 16-byte vectors of every layer's rows
// of K and V (layer l at k + l * layer_vec, v + l * layer_vec); blockIdx.y
// walks the layers.
__global__ void __launch_bounds__(256) fill_kernel(u32x4* __restrict__ k, u32x4* __restrict__ v,
                                                   int32_t n_layers, int64_t layer_vec, int64_t n_vec,
                                                   uint32_t fill_word) {
  const u32x4 fill = {fill_word, fill_word, fill_word, fill_word};
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int32_t layer = blockIdx.y; layer < n_layers; layer += gridDim.y) {
    u32x4* kl = k + layer * layer_vec;
    u32x4* vl = v + layer * layer_vec;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_vec; i += stride) {
      __builtin_nontemporal_store(fill, kl + i);
      __builtin_nontemporal_store(fill, vl + i);
    }
  }
}

// The step's mask, mask[b * ld + j] for j in [0, L + T): a live row (span n)
// is 1 on [L - n, L] outside its holes, a row prefilled this step (prompt p)
// on [L + T - p, L + T), a free row nowhere.  One block row per slot, 4 bytes
// per thread (one 4-byte store where the row allows it).
struct MaskArgs {
  uint8_t* mask;
  int64_t ld, L;
  int32_t batch, T;
  int32_t lens[512];      // span; 0 free; -p prefilled this step with a prompt of p tokens
  uint8_t first[512];     // index of the row's first hole
  HoleList holes;
};

__global__ void __launch_bounds__(256) mask_kernel(const MaskArgs a) {
  const int b = blockIdx.y;
  const int32_t n = a.lens[b];
  const int64_t W = a.L + a.T;
  int64_t lo, hi;                                   // the ones before holes: [lo, hi)
  if (n > 0) {
    lo = a.L - n;
    hi = a.L + 1;
  } else if (n < 0) {
    lo = W + n;
    hi = W;
  } else {
    lo = hi = 0;
  }
  const int k0 = n > 0 ? a.first[b] : a.holes.n;
  const int nh = a.holes.n;
  uint8_t* row = a.mask + (int64_t)b * a.ld;
  for (int64_t j0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4; j0 < W;
       j0 += (int64_t)gridDim.x * blockDim.x * 4) {
    // The row's holes are sorted and disjoint: the first one ending past j0,
    // by bisection, then forward as j advances.
    int k = k0, k_hi = nh;
    while (k < k_hi) {
      const int mid = (k + k_hi) / 2;
      if (a.holes.col[mid][1] <= j0) k = mid + 1;
      else k_hi = mid;
    }
    uint32_t word = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t j = j0 + e;
      while (k < nh && a.holes.col[k][1] <= j) ++k;
      const bool one = j >= lo && j < hi && !(k < nh && j >= a.holes.col[k][0]);
      word |= (uint32_t)one << (8 * e);
    }
    if (j0 + 4 <= W && (reinterpret_cast<uintptr_t>(row + j0) & 3) == 0) {
      *reinterpret_cast<uint32_t*>(row + j0) = word;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (j0 + e < W) row[j0 + e] = (uint8_t)(word >> (8 * e));
    }
  }
}

}  // namespace baton
