// Masked batched decode attention over the aligned ring cache, split over the
// sequence ("split-K") so that long and skewed rows spread over all CUs.
//
// Work item = (slot b, split c) x kv-head h: the tokens t in
// [c*S, min((c+1)*S, len_b+1)) of row (layer, b, h), where token t < len_b is
// cache column L - len_b + t and token len_b is the current token (k_new/v_new,
// appended to the cache by the item that holds it).  Placeholder columns are
// never addressed.  One wave per item: a token row of D elements is spread
// over LPT = D*elem/16 lanes (16 bytes each), so one wave instruction reads
// TPI = 64/LPT whole token rows; each of those TPI lane groups keeps its own
// online-softmax state (max m, sum l, weighted values acc) over the tokens it
// reads, and the groups merge once at the end of the item.  Items of a row
// that has one item write the output; otherwise they write (m, l, acc)
// partials that the combine kernel merges with the log-sum-exp rescale.
// Exponentials are base 2 with scale*log2(e) folded into q.
#pragma once

#include "common.hpp"

namespace baton {

constexpr int kMetaThreads = 512;   // == BATON_MAX_BATCH

struct MetaArgs {
  int32_t batch;
  int32_t split;                    // tokens per item
  int32_t lens[kMetaThreads];
};

// Builds the per-step work list in the workspace: lens[b], item_start[b]
// (exclusive prefix of items per row, batch + 1 entries) and items[] = (b, c).
__global__ void __launch_bounds__(kMetaThreads) meta_kernel(const MetaArgs a, int32_t* ws_lens,
                                                            int32_t* ws_item_start,
                                                            int2* ws_items) {
  __shared__ int32_t scan[kMetaThreads];
  const int b = threadIdx.x;
  const int32_t n = b < a.batch ? a.lens[b] : 0;
  const int32_t cnt = n > 0 ? (n + a.split) / a.split : 0;   // ceil((n + 1) / split)
  scan[b] = cnt;
  __syncthreads();
  for (int off = 1; off < kMetaThreads; off <<= 1) {
    const int32_t add = b >= off ? scan[b - off] : 0;
    __syncthreads();
    scan[b] += add;
    __syncthreads();
  }
  const int32_t excl = scan[b] - cnt;
  if (b < a.batch) {
    ws_lens[b] = n;
    ws_item_start[b] = excl;
    if (b == a.batch - 1) ws_item_start[a.batch] = scan[b];
    for (int32_t c = 0; c < cnt; ++c) ws_items[excl + c] = make_int2(b, c);
  }
}

struct AttnArgs {
  const uint32_t* k;         // ring buffers (whole cache), 32-bit words
  uint32_t* v;
  uint32_t* k_w;             // same as k, writable (append)
  const uint32_t* q;         // [batch][n_q_heads][D]
  const uint32_t* knew;      // [batch][n_kv_heads][D]
  const uint32_t* vnew;
  uint32_t* out;             // [batch][n_q_heads][D]
  const int32_t* lens;       // workspace
  const int32_t* item_start;
  const int2* items;
  float* partial;            // [n_kv_heads][n_items][G][D + 4]
  int64_t cap, base, L;
  int32_t layer, batch, n_kv_heads, split, n_items;
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

template <typename T, int D, int G, int U>
__global__ void __launch_bounds__(kWave) attn_kernel(const AttnArgs a) {
  using Geo = Geometry<T, D>;
  constexpr int EPL = Geo::kEpl, LPT = Geo::kLpt, TPI = Geo::kTpi, VPT = Geo::kVpt;
  constexpr int REC = D + 4;   // floats per partial record
  const int item = blockIdx.x;
  const int h = blockIdx.y;
  const int lane = threadIdx.x;
  const int r = lane / LPT;        // token row within an instruction
  const int cl = lane % LPT;       // 16-byte slice of the row

  const int2 bc = a.items[item];
  const int b = bc.x, c = bc.y;
  const int32_t n = a.lens[b];     // cached tokens; token n is the current one
  const int32_t t_begin = c * a.split;
  const int32_t t_end = min(t_begin + a.split, n + 1);
  const bool whole_row = (t_begin == 0) && (t_end == n + 1);

  const int64_t row = ((int64_t)a.layer * a.batch + b) * a.n_kv_heads + h;
  const u32x4* Krow = reinterpret_cast<const u32x4*>(a.k) + row * a.cap * VPT;
  const u32x4* Vrow = reinterpret_cast<const u32x4*>(a.v) + row * a.cap * VPT;
  const int64_t start = ring_add(a.base, a.L - n, a.cap);   // physical column of token 0
  const u32x4* knew = reinterpret_cast<const u32x4*>(a.knew) + ((int64_t)b * a.n_kv_heads + h) * VPT;
  const u32x4* vnew = reinterpret_cast<const u32x4*>(a.vnew) + ((int64_t)b * a.n_kv_heads + h) * VPT;

  // Query slices of the G heads that share kv-head h, pre-scaled.
  float qf[G][EPL];
#pragma unroll
  for (int gi = 0; gi < G; ++gi) {
    const u32x4 w = reinterpret_cast<const u32x4*>(a.q)[(((int64_t)b * a.n_kv_heads + h) * G + gi) * VPT + cl];
    Lane16<T>::widen(w, qf[gi]);
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

  for (int32_t tt = t_begin; tt < t_end; tt += TPI * U) {
    u32x4 kw[U], vw[U];
    bool valid[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int32_t t = tt + u * TPI + r;
      valid[u] = t < t_end;
      kw[u] = u32x4{0, 0, 0, 0};
      vw[u] = u32x4{0, 0, 0, 0};
      if (valid[u]) {
        if (t < n) {
          const int64_t col = ring_add(start, t, a.cap);
          kw[u] = __builtin_nontemporal_load(Krow + col * VPT + cl);
          vw[u] = __builtin_nontemporal_load(Vrow + col * VPT + cl);
        } else {
          kw[u] = knew[cl];
          vw[u] = vnew[cl];
        }
      }
    }
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
      const float alpha = exp2f(m[gi] - ref);
      l[gi] *= alpha;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[gi][e] *= alpha;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float p = exp2f(s[u][gi] - ref);
        l[gi] += p;
        float vf[EPL];
        Lane16<T>::widen(vw[u], vf);
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[gi][e] = fmaf(p, vf[e], acc[gi][e]);
      }
      m[gi] = mt;
    }
  }

  // The current token goes into the cache as column L (once per row).
  if (n >= t_begin && n < t_end && (n - t_begin) % TPI == r) {
    const int64_t col = ring_add(start, n, a.cap);
    reinterpret_cast<u32x4*>(a.k_w)[row * a.cap * VPT + col * VPT + cl] = knew[cl];
    reinterpret_cast<u32x4*>(a.v)[row * a.cap * VPT + col * VPT + cl] = vnew[cl];
  }

  // Merge the TPI lane groups.
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

  if (r != 0) return;
  if (whole_row) {
#pragma unroll
    for (int gi = 0; gi < G; ++gi) {
      const float inv = 1.f / l[gi];
      float o[EPL];
#pragma unroll
      for (int e = 0; e < EPL; ++e) o[e] = acc[gi][e] * inv;
      reinterpret_cast<u32x4*>(a.out)[(((int64_t)b * a.n_kv_heads + h) * G + gi) * VPT + cl] =
          Lane16<T>::narrow(o);
    }
  } else {
#pragma unroll
    for (int gi = 0; gi < G; ++gi) {
      float* rec = a.partial + (((int64_t)h * a.n_items + item) * G + gi) * REC;
#pragma unroll
      for (int e = 0; e < EPL; ++e) rec[cl * EPL + e] = acc[gi][e];
      if (cl == 0) {
        rec[D] = m[gi];
        rec[D + 1] = l[gi];
      }
    }
  }
}

// One wave per (slot, kv-head): zeros for a free slot, nothing for a slot with
// one item, the log-sum-exp merge of the partials otherwise.
template <typename T, int D, int G>
__global__ void __launch_bounds__(kWave) combine_kernel(const AttnArgs a) {
  constexpr int REC = D + 4;
  constexpr int PER = D / kWave;   // elements per lane (1 or 2)
  const int b = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  const int32_t i0 = a.item_start[b], i1 = a.item_start[b + 1];
  if (i1 - i0 == 1) return;
  for (int gi = 0; gi < G; ++gi) {
    float o[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) o[e] = 0.f;
    if (i1 > i0) {
      const float* base = a.partial + ((int64_t)h * a.n_items * G + gi) * REC;
      float mm = -INFINITY;
      for (int32_t i = i0; i < i1; ++i) mm = fmaxf(mm, base[(int64_t)i * G * REC + D]);
      float l = 0.f;
      for (int32_t i = i0; i < i1; ++i) {
        const float* rec = base + (int64_t)i * G * REC;
        const float w = rec[D] == -INFINITY ? 0.f : exp2f(rec[D] - mm);
        l += w * rec[D + 1];
#pragma unroll
        for (int e = 0; e < PER; ++e) o[e] = fmaf(w, rec[lane * PER + e], o[e]);
      }
      const float inv = 1.f / l;
#pragma unroll
      for (int e = 0; e < PER; ++e) o[e] *= inv;
    }
    const int64_t obase = (((int64_t)b * a.n_kv_heads + h) * G + gi) * D + lane * PER;
    if constexpr (T::kBytes == 4) {
#pragma unroll
      for (int e = 0; e < PER; ++e) a.out[obase + e] = __float_as_uint(o[e]);
    } else {
      uint16_t* out16 = reinterpret_cast<uint16_t*>(a.out);
#pragma unroll
      for (int e = 0; e < PER; ++e) out16[obase + e] = (uint16_t)f32_to_bf16_rne(o[e]);
    }
  }
}

}  // namespace baton
