// Causal attention of the queries prefilled inside the batch, for a step
// without prefill/decode separation: a new query's prompt of p tokens sits at
// input positions T - p .. T - 1 of its row (q [batch][T][n_q_heads][D],
// k_new / v_new [batch][T][n_kv_heads][D]); prompt position i attends over
// prompt positions 0 .. i -- the rest of its row is masked -- and every prompt
// position's key and value is appended to the cache as column L + T - p + i.
// The other rows of the step are decoded by the work-item kernels.
//
// Work: one wave per (tile of prompt positions, query head); the tiles of the
// prefilled queries are numbered consecutively, a query's longest tiles (the
// last positions, which see the most keys) first.  Keys and values come
// straight from k_new / v_new (the whole prompt is read by every tile of a
// head, through the caches).  The first query head of each kv-head appends
// its tile's positions.
#pragma once

#include "common.hpp"
#include "decode_attn.hpp"
#include "decode_attn_mfma.hpp"

namespace baton {

constexpr int kMaxPrefill = 64;   // == BATON_MAX_PREFILL

struct PrefillArgs {
  uint32_t* k;              // ring buffers (appended to)
  uint32_t* v;
  const uint32_t* q;        // [batch][T][n_q_heads][D]
  const uint32_t* knew;     // [batch][T][n_kv_heads][D]
  const uint32_t* vnew;
  uint32_t* out;            // [batch][T][n_q_heads][D]
  int64_t cap, base, L;
  int32_t T, layer, batch, n_kv_heads, n_ins;
  float qscale;             // scale * log2(e)
  int32_t slot[kMaxPrefill];
  int32_t plen[kMaxPrefill];
  int32_t tile_end[kMaxPrefill];   // inclusive prefix of tiles over the prefilled queries
};

// The prefilled query and tile of block x; tiles are handed out last first.
__device__ __forceinline__ void prefill_tile(const PrefillArgs& a, int32_t& i, int32_t& tile) {
  const int32_t g = blockIdx.x;
  i = 0;
  while (i < a.n_ins - 1 && g >= a.tile_end[i]) ++i;
  tile = a.tile_end[i] - 1 - g;   // the query's tiles, counted from its last one
}

// Appends prompt positions [t0, t0 + n) of kv-head h (all lanes of the wave).
template <int VPT>
__device__ __forceinline__ void prefill_append(const PrefillArgs& a, int b, int h, int32_t p,
                                               int64_t row0, int32_t t0, int32_t n, int lane) {
  const int64_t ring_row = ((int64_t)a.layer * a.batch + b) * a.n_kv_heads + h;
  u32x4* rk = reinterpret_cast<u32x4*>(a.k) + ring_row * a.cap * VPT;
  u32x4* rv = reinterpret_cast<u32x4*>(a.v) + ring_row * a.cap * VPT;
  const u32x4* kin = reinterpret_cast<const u32x4*>(a.knew);
  const u32x4* vin = reinterpret_cast<const u32x4*>(a.vnew);
  const int64_t c0 = a.base + a.L + a.T - p;   // < 2 * cap: base < cap, L + T <= cap
  for (int idx = lane; idx < n * VPT; idx += kWave) {
    const int32_t t = t0 + idx / VPT;
    const int e = idx % VPT;
    int64_t col = c0 + t;
    col = col >= a.cap ? col - a.cap : col;
    const int64_t src = ((row0 + t) * a.n_kv_heads + h) * VPT + e;
    rk[col * VPT + e] = kin[src];
    rv[col * VPT + e] = vin[src];
  }
}

// bf16 on the matrix cores: 16 prompt positions per wave as the 16 columns of
// mfma_block's query operand, 32 keys per iteration, a causal mask per lane
// (lane l scores the keys of position l % 16).
template <int D, int G>
__global__ void __launch_bounds__(kWave) prefill_mfma_kernel(const PrefillArgs a) {
  using Geo = MfmaGeo<D>;
  constexpr int VPT = Geo::kVpt, KK = Geo::kKk, DT = Geo::kDt;
  __shared__ __attribute__((aligned(16))) uint8_t lds[32 * Geo::kLdsRow];
  const int hq = blockIdx.y, h = hq / G, lane = threadIdx.x;
  const int g4 = lane / 16, c16 = lane % 16;
  int32_t ins, tile;
  prefill_tile(a, ins, tile);
  const int b = a.slot[ins];
  const int32_t p = a.plen[ins];
  const int32_t i0 = tile * 16;
  const int64_t row0 = (int64_t)b * a.T + (a.T - p);   // input row of prompt position 0
  const int nkv = a.n_kv_heads, nq = nkv * G;
  const u32x4* qin = reinterpret_cast<const u32x4*>(a.q);
  const u32x4* kin = reinterpret_cast<const u32x4*>(a.knew);
  const u32x4* vin = reinterpret_cast<const u32x4*>(a.vnew);
  const u32x4 zero = {0, 0, 0, 0};

  const int32_t qi = i0 + c16;                          // this lane's query position
  bf16x8 qb[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk)
    qb[kk] = as_bf16x8(qi < p ? qin[((row0 + qi) * nq + hq) * VPT + kk * 4 + g4] : zero);

  float m = -INFINITY, lsum = 0.f;
  f32x4 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int32_t last = min(i0 + 15, p - 1);            // last position of the tile
  const int tau = (c16 / 4) + 4 * (c16 % 4);          // token of this lane's key row in a tile
  for (int32_t tt = 0; tt <= last; tt += 32) {
    u32x4 kA[KK], kB[KK], vw[Geo::kVLoads];
    const int32_t ta = tt + tau, tb = tt + 16 + tau;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      kA[kk] = ta < p ? kin[((row0 + ta) * nkv + h) * VPT + kk * 4 + g4] : zero;
      kB[kk] = tb < p ? kin[((row0 + tb) * nkv + h) * VPT + kk * 4 + g4] : zero;
    }
#pragma unroll
    for (int u = 0; u < Geo::kVLoads; ++u) {
      const int32_t t = tt + u * Geo::kTpiV + lane / VPT;
      vw[u] = t < p ? vin[((row0 + t) * nkv + h) * VPT + lane % VPT] : zero;
    }
    const int32_t lim = qi < p ? qi - tt : -1;         // keys tt .. tt + lim are visible
    const uint32_t mask = lim >= 31 ? 0xFFFFFFFFu : (lim < 0 ? 0u : ((2u << lim) - 1u));
    mfma_block<D, G>(kA, kB, vw, qb, mask, a.qscale, lds, m, lsum, o, lane);
  }

  // Row sums over the four lane groups; lane l's output rows are positions i0 + 4*g4 + r.
  lsum += __shfl_xor(lsum, 16, kWave);
  lsum += __shfl_xor(lsum, 32, kWave);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int qr = 4 * g4 + r;
    const float lr = __shfl(lsum, qr, kWave);
    if (i0 + qr < p) {
      const float inv = 1.f / lr;
      uint16_t* o16 = reinterpret_cast<uint16_t*>(a.out) + ((row0 + i0 + qr) * nq + hq) * D;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o16[16 * dt + c16] = (uint16_t)f32_to_bf16_rne(o[dt][r] * inv);
    }
  }
  if (hq % G == 0) prefill_append<VPT>(a, b, h, p, row0, i0, min(16, p - i0), lane);
}

// Any element type on the vector ALUs: a prompt position per lane group (LPT
// lanes, 16 bytes each), TPI positions per wave, the keys one at a time.
template <typename T, int D, int G>
__global__ void __launch_bounds__(kWave) prefill_valu_kernel(const PrefillArgs a) {
  using Geo = Geometry<T, D>;
  constexpr int EPL = Geo::kEpl, LPT = Geo::kLpt, TPI = Geo::kTpi, VPT = Geo::kVpt;
  const int hq = blockIdx.y, h = hq / G, lane = threadIdx.x;
  const int r = lane / LPT, cl = lane % LPT;
  int32_t ins, tile;
  prefill_tile(a, ins, tile);
  const int b = a.slot[ins];
  const int32_t p = a.plen[ins];
  const int32_t i0 = tile * TPI;
  const int64_t row0 = (int64_t)b * a.T + (a.T - p);
  const int nkv = a.n_kv_heads, nq = nkv * G;
  const u32x4* kin = reinterpret_cast<const u32x4*>(a.knew);
  const u32x4* vin = reinterpret_cast<const u32x4*>(a.vnew);

  const int32_t qi = i0 + r;                           // this lane group's position
  float qf[EPL];
  {
    const u32x4 w = qi < p ? reinterpret_cast<const u32x4*>(a.q)[((row0 + qi) * nq + hq) * VPT + cl]
                           : u32x4{0, 0, 0, 0};
    Lane16<T>::widen(w, qf);
#pragma unroll
    for (int e = 0; e < EPL; ++e) qf[e] *= a.qscale;
  }
  float m = -INFINITY, l = 0.f, acc[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) acc[e] = 0.f;
  const int32_t last = min(i0 + TPI - 1, p - 1);
  for (int32_t t = 0; t <= last; ++t) {
    const int64_t src = ((row0 + t) * nkv + h) * VPT + cl;
    float kf[EPL], vf[EPL];
    Lane16<T>::widen(kin[src], kf);
    Lane16<T>::widen(vin[src], vf);
    float d = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) d = fmaf(qf[e], kf[e], d);
    d = group_sum<LPT>(d);
    if (t <= qi) {
      const float mn = fmaxf(m, d);
      const float alpha = exp2f(m - mn);   // m = -inf at the first key: 0
      const float pw = exp2f(d - mn);
      l = l * alpha + pw;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[e] = fmaf(pw, vf[e], acc[e] * alpha);
      m = mn;
    }
  }
  if (qi < p) {
    const float inv = 1.f / l;
    float o[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[e] = acc[e] * inv;
    reinterpret_cast<u32x4*>(a.out)[((row0 + qi) * nq + hq) * VPT + cl] = Lane16<T>::narrow(o);
  }
  if (hq % G == 0) prefill_append<VPT>(a, b, h, p, row0, i0, min(TPI, p - i0), lane);
}

}  // namespace baton
