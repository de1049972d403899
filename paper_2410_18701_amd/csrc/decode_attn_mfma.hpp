// Grouped-query decode attention on the matrix cores (bf16, G = 2, 4 or 8
// query heads per kv head).  With G query heads sharing a key row the work is
// G times denser than multi-head attention, enough to make the VALU the
// limiter; here QK^T and PV run as v_mfma_f32_16x16x32_bf16 tiles.
//
// Per iteration a wave takes 32 tokens of its work item as two 16-token tiles.
//  * QK^T: A = 16 key rows x 32 d (lane l supplies row l%16, d-group l/16),
//    B = the G query heads padded to 16 columns, D = head_dim/32 MFMAs.
//    The A row of lane l is token tau(l%16) with tau(4g + r) = g + 4r, so the
//    result row 4g + r (held by lane group g, register r) is token g + 4r.
//  * softmax: lane l holds head l%16's scores of 8 tokens; the running max is
//    shared by the four lane groups (all of them accumulate into the same
//    output tile), exponentials are base 2, P is rounded to bf16.
//  * PV, transposed (O^T = V^T P^T): B = P^T (32 tokens x 16 heads, lane l:
//    head l%16, its own 8 tokens as k = 8*(l/16) + e), A = V^T (16 d x 32
//    tokens) per 16-column slice of head_dim, so lane l accumulates output
//    columns 16*dt + 4*(l/16) + r of head l%16 and rescales with its own
//    factor.  K and V are both loaded as whole rows (coalesced, 1 KB per
//    load instruction) and staged in LDS row by row; K is read back as the A
//    operand (16 bytes per lane), V transposed, 2 bytes per lane; the token
//    order above makes the four lane groups of one V read hit consecutive
//    rows, i.e. disjoint banks.
// The current token (k_new, v_new) is a one-token tile of its own.  As in the
// VALU kernel, a workgroup of NW waves takes one work item, each wave an equal
// contiguous share of its tokens, and the waves merge through LDS; partial
// records and outputs have the layout of the VALU kernel, so combine_kernel
// merges both.
#pragma once

#include "common.hpp"
#include "decode_attn.hpp"

namespace baton {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8 as_bf16x8(const u32x4& w) { return __builtin_bit_cast(bf16x8, w); }

template <int D>
struct MfmaGeo {
  static constexpr int kVpt = D / 8;              // 16-byte vectors per token row
  static constexpr int kTpiV = kWave / kVpt;      // token rows per V load instruction
  static constexpr int kVLoads = 32 / kTpiV;      // V loads per lane per 32 tokens
  static constexpr int kKk = D / 32;              // QK MFMAs per tile
  static constexpr int kDt = D / 16;              // PV MFMAs (16-column slices)
  static constexpr int kLdsRow = D * 2 + 32;      // padded LDS row (bank spread)
};

// One 32-token block: scores, online softmax, PV.  kw, vw: this lane's K and V
// vectors, read as whole rows (lane l: 16 bytes at (l % kVpt) * 16 of token
// u * kTpiV + l / kVpt) -- contiguous 1 KB per load instruction, which the
// DRAM serves about 7% faster than the A operand's own pattern (16 rows x 64
// bytes per instruction); valid_mask: bit t set when token t (0..31) of the
// block takes part.  Both go through LDS (row t holds token t of the block):
// the key tiles are read back as A operands, the values transposed.
template <int D, int G>
__device__ __forceinline__ void mfma_block(const u32x4 (&kw)[MfmaGeo<D>::kVLoads],
                                           const u32x4 (&vw)[MfmaGeo<D>::kVLoads],
                                           const bf16x8 (&qb)[D / 32], uint32_t valid_mask,
                                           float qscale, uint8_t* lds_k, uint8_t* lds, float& m,
                                           float& lsum, f32x4 (&o)[D / 16], int lane) {
  using Geo = MfmaGeo<D>;
  const int g4 = lane / 16, c16 = lane % 16;
#pragma unroll
  for (int u = 0; u < Geo::kVLoads; ++u) {
    const int t = u * Geo::kTpiV + lane / Geo::kVpt;
    *reinterpret_cast<u32x4*>(lds_k + t * Geo::kLdsRow + (lane % Geo::kVpt) * 16) = kw[u];
    *reinterpret_cast<u32x4*>(lds + t * Geo::kLdsRow + (lane % Geo::kVpt) * 16) = vw[u];
  }
  // The key tiles as A operands: lane l supplies row tau(l % 16) of each tile
  // (tau(4g + r) = g + 4r) and its d-group l / 16 of each 32-wide step.
  const int tau = (c16 / 4) + 4 * (c16 % 4);
  // Scores of the two tiles: s[r] for token g4 + 4r, s[4 + r] for token 16 + g4 + 4r.
  f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kk = 0; kk < Geo::kKk; ++kk) {
    const u32x4 ka = *reinterpret_cast<const u32x4*>(lds_k + tau * Geo::kLdsRow + (kk * 4 + g4) * 16);
    const u32x4 kb = *reinterpret_cast<const u32x4*>(lds_k + (16 + tau) * Geo::kLdsRow + (kk * 4 + g4) * 16);
    sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ka), qb[kk], sa, 0, 0, 0);
    sb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kb), qb[kk], sb, 0, 0, 0);
  }
  float s[8];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    s[r] = ((valid_mask >> (g4 + 4 * r)) & 1u) ? sa[r] * qscale : -INFINITY;
    s[4 + r] = ((valid_mask >> (16 + g4 + 4 * r)) & 1u) ? sb[r] * qscale : -INFINITY;
  }
  float mx = s[0];
#pragma unroll
  for (int e = 1; e < 8; ++e) mx = fmaxf(mx, s[e]);
  mx = max_over_groups(mx);
  const float mn = fmaxf(m, mx);
  const float ref = mn == -INFINITY ? 0.f : mn;
  const float alpha = exp2f(m - ref);
  bf16x8 pa;
  float psum = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const __bf16 pb = (__bf16)exp2f(s[e] - ref);
    pa[e] = pb;
    psum += (float)pb;
  }
  lsum = lsum * alpha + psum;
  m = mn;
  // Rescale the output column this lane holds (head c16).
#pragma unroll
  for (int dt = 0; dt < Geo::kDt; ++dt) o[dt] *= alpha;
  // PV, transposed: A = V^T (row 16*dt + c16, keys token(k), k = 8*g4 + e),
  // B = P^T (this lane's own probabilities); lane l accumulates output
  // columns 16*dt + 4*g4 + r of head c16.
#pragma unroll
  for (int dt = 0; dt < Geo::kDt; ++dt) {
    bf16x8 vb;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int t = e < 4 ? g4 + 4 * e : 16 + g4 + 4 * (e - 4);
      vb[e] = *reinterpret_cast<const __bf16*>(lds + t * Geo::kLdsRow + (16 * dt + c16) * 2);
    }
    o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vb, pa, o[dt], 0, 0, 0);
  }
}

#ifndef BATON_MFMA_WAVES_PER_EU
#define BATON_MFMA_WAVES_PER_EU 0   // 0: compiler's choice
#endif

template <int D, int G, int NW>
__global__ void __launch_bounds__(kWave * NW)
#if BATON_MFMA_WAVES_PER_EU > 0
__attribute__((amdgpu_waves_per_eu(BATON_MFMA_WAVES_PER_EU)))
#endif
attn_mfma_kernel(const AttnArgs a) {
  using Geo = MfmaGeo<D>;
  constexpr int VPT = Geo::kVpt, KK = Geo::kKk, DT = Geo::kDt, REC = D + 4;
  // Per wave: the K and V staging of a block; after the wave's last block its
  // K staging holds its G x D accumulator for the workgroup's merge.
  __shared__ __attribute__((aligned(16))) uint8_t lds_k[NW][32 * Geo::kLdsRow];
  __shared__ __attribute__((aligned(16))) uint8_t lds_v[NW][32 * Geo::kLdsRow];
  __shared__ float sm_m[NW][G], sm_l[NW][G];
  static_assert(G * D * 4 <= 32 * Geo::kLdsRow, "merge area");
  int32_t item, h;
  const Item desc = work_unit(a, item, h);
  const int tid = threadIdx.x;
  // wave of the workgroup, as a scalar: the loop bounds derived from it are uniform
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave), lane = tid % kWave;
  const int g4 = lane / 16, c16 = lane % 16;
  uint8_t* lds = lds_v[w];
  uint8_t* ldk = lds_k[w];

  const int4 it = desc.span;
  const int4 rw = desc.row;
  const int b = it.x;
  const int32_t n = it.w;
  const int64_t bt = (int64_t)b * a.tw;   // input row of the slot's position 0
  uint32_t* outw = a.out + ((bt * a.n_kv_heads + h) * G) * (D / 2);
  if (n < 0) {                       // free slot: zero output rows
    for (int v = tid; v < G * VPT; v += NW * kWave) reinterpret_cast<u32x4*>(outw)[v] = u32x4{0, 0, 0, 0};
    return;
  }
  int32_t t_begin, t_end;            // this wave's share of the item's tokens
  wave_share<NW, 32>(it.y, it.z, w, t_begin, t_end);
  const int64_t row = (int64_t)b * a.n_kv_heads + h;   // within the layer's rows
  constexpr uint32_t ROWB = VPT * 16;
  const uint32_t ring_bytes = (uint32_t)a.cap * ROWB;
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(a.k) + row * a.cap * VPT * 4, 0,
                                        ring_bytes, kBufferWord3);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc(a.v + row * a.cap * VPT * 4, 0, ring_bytes, kBufferWord3);
  const uint32_t start = (uint32_t)ring_add(a.base, a.L - n, a.cap);
  const uint32_t cap = (uint32_t)a.cap;

  // Query heads as the B operand: column c16 = head c16 (zero beyond G).
  bf16x8 qb[KK];
  const u32x4* qrow = reinterpret_cast<const u32x4*>(a.q) + ((bt * a.n_kv_heads + h) * G) * VPT;
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    const u32x4 qw = c16 < G ? qrow[c16 * VPT + kk * 4 + g4] : u32x4{0, 0, 0, 0};
    qb[kk] = as_bf16x8(qw);
  }

  float m = -INFINITY, lsum = 0.f;
  f32x4 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const bool gathered = (rw.w & kGathered) != 0;
  if (gathered) {
    // A gathered item: its share of the listed tokens (short runs of a
    // holey row), 32 per block; the token indices first, then the rows.
    for (int32_t i0 = t_begin; i0 < t_end; i0 += 32) {
      int32_t tok[Geo::kVLoads];
#pragma unroll
      for (int u = 0; u < Geo::kVLoads; ++u) {
        const int32_t i = i0 + u * Geo::kTpiV + lane / VPT;
        tok[u] = i < t_end ? a.gather[i] : -1;
      }
      u32x4 kw[Geo::kVLoads], vw[Geo::kVLoads];
#pragma unroll
      for (int u = 0; u < Geo::kVLoads; ++u) {
        uint32_t col = start + (uint32_t)max(tok[u], 0);
        col = col >= cap ? col - cap : col;
        const uint32_t off = tok[u] >= 0 ? col * ROWB + (lane % VPT) * 16u : 0x80000000u;
        kw[u] = load16(rk, off);
        vw[u] = load16(rv, off);
      }
      const int32_t nvalid = min(32, t_end - i0);
      const uint32_t mask = nvalid >= 32 ? 0xFFFFFFFFu : ((1u << nvalid) - 1u);
      mfma_block<D, G>(kw, vw, qb, mask, a.qscale, ldk, lds, m, lsum, o, lane);
    }
  } else {
    const int32_t c_end = min(t_end, n);
    for (int32_t tt = t_begin; tt < c_end; tt += 32) {
      u32x4 kw[Geo::kVLoads], vw[Geo::kVLoads];
#pragma unroll
      for (int u = 0; u < Geo::kVLoads; ++u) {
        const int32_t t = tt + u * Geo::kTpiV + lane / VPT;
        uint32_t col = start + (uint32_t)t;
        col = col >= cap ? col - cap : col;
        // past the end: an offset beyond the buffer, which loads zeros
        const uint32_t off = t < c_end ? col * ROWB + (lane % VPT) * 16u : 0x80000000u;
        kw[u] = load16(rk, off);
        vw[u] = load16(rv, off);
      }
      const int32_t nvalid = min(32, c_end - tt);
      const uint32_t mask = nvalid >= 32 ? 0xFFFFFFFFu : ((1u << nvalid) - 1u);
      mfma_block<D, G>(kw, vw, qb, mask, a.qscale, ldk, lds, m, lsum, o, lane);
    }
  }

  // The current token, a one-token tile read from k_new / v_new, and its
  // append (of a gathered item, by its first wave).
  if (gathered ? (rw.w & kCurrent) != 0 && w == 0 : n >= t_begin && n < t_end) {
    const u32x4* knew = reinterpret_cast<const u32x4*>(a.knew) + (bt * a.n_kv_heads + h) * VPT;
    const u32x4* vnew = reinterpret_cast<const u32x4*>(a.vnew) + (bt * a.n_kv_heads + h) * VPT;
    u32x4 kw[Geo::kVLoads], vw[Geo::kVLoads];   // token 0 of the block; the other rows zero
#pragma unroll
    for (int u = 0; u < Geo::kVLoads; ++u) {
      kw[u] = (u == 0 && lane < VPT) ? knew[lane] : u32x4{0, 0, 0, 0};
      vw[u] = (u == 0 && lane < VPT) ? vnew[lane] : u32x4{0, 0, 0, 0};
    }
    mfma_block<D, G>(kw, vw, qb, 1u, a.qscale, ldk, lds, m, lsum, o, lane);
    if (lane < VPT) {
      const uint32_t col = (uint32_t)ring_add(start, n, a.cap);
      reinterpret_cast<u32x4*>(a.k_w)[row * a.cap * VPT + (int64_t)col * VPT + lane] = knew[lane];
      reinterpret_cast<u32x4*>(a.v)[row * a.cap * VPT + (int64_t)col * VPT + lane] = vnew[lane];
    }
  }

  // Sums over the four lane groups; lane l holds output columns
  // 16*dt + 4*g4 + r of head c16.  The wave's state goes to LDS for the
  // workgroup's merge.
  lsum = sum_over_groups(lsum);
  if (c16 < G) {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int r = 0; r < 4; ++r) reinterpret_cast<float*>(ldk)[c16 * D + 16 * dt + 4 * g4 + r] = o[dt][r];
    if (g4 == 0) {
      sm_m[w][c16] = m;
      sm_l[w][c16] = lsum;
    }
  }
  __syncthreads();
  float* rec0 = a.partial + (((int64_t)h * a.n_items + item) * G) * REC;
  wg_merge_write<BF16Tag, D, G, NW>(sm_m, sm_l, reinterpret_cast<const float*>(&lds_k[0][0]),
                                    32 * Geo::kLdsRow / 4, rw.y == 1, outw, rec0, tid);
}

}  // namespace baton
