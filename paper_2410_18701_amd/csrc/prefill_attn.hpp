// Causal attention of the queries prefilled inside the batch, for a step
// without prefill/decode separation: a new query's prompt of p tokens sits at
// input positions T - p .. T - 1 of its row (q [batch][T][n_q_heads][D],
// k_new / v_new [batch][T][n_kv_heads][D]); prompt position i attends over
// prompt positions 0 .. i -- the rest of its row is masked -- and every prompt
// position's key and value is appended to the cache as column L + T - p + i.
// The other rows of the step are decoded by the work-item kernels.
//
// Work: one workgroup per (tile of prompt positions, query head); the tiles
// of the prefilled queries are numbered consecutively, a query's longest
// tiles (the last positions, which see the most keys) first.  Keys and values
// come straight from k_new / v_new (the prompt is read by every tile of a
// head, through the caches).  The appends to the cache run in workgroups of
// their own, one per (tile, kv-head), after all the attention workgroups in
// the grid of prefill_fa_kernel (bf16, on the matrix cores): short ones, they
// fill the end of the launch instead of lengthening every attention
// workgroup by a load and a store of its tile; in prefill_valu_kernel (fp32,
// the vector ALUs) the first query head of each kv-head appends its tile.
#pragma once

#include "common.hpp"
#include "decode_attn.hpp"
#include "decode_attn_mfma.hpp"   // bf16x8, f32x4, as_bf16x8

namespace baton {

constexpr int kMaxPrefill = 64;   // == BATON_MAX_PREFILL

struct PrefillArgs {
  uint32_t* k;              // the layer's ring rows [batch][n_kv_heads][cap][D] (appended to)
  uint32_t* v;
  const uint32_t* q;        // [batch][T][n_q_heads][D]
  const uint32_t* knew;     // [batch][T][n_kv_heads][D]
  const uint32_t* vnew;
  uint32_t* out;            // [batch][T][n_q_heads][D]
  int64_t cap, base, L;
  int32_t T, batch, n_kv_heads, n_ins;
  int32_t n_tiles;          // tiles over all prefilled queries (per query head)
  int32_t unit_heads;       // query heads that read the same keys (G), or 1
  int32_t xcd_map;          // 1: keep each unit's workgroups on one XCD (units % 8 == 0)
  int32_t n_attn;           // attention workgroups (n_tiles x query heads); the matrix-core
                            // kernel's grid then has n_tiles x n_kv_heads append workgroups
  float qscale;             // scale * log2(e)
  int32_t slot[kMaxPrefill];
  int32_t plen[kMaxPrefill];
  int32_t tile_end[kMaxPrefill];   // inclusive prefix of tiles over the prefilled queries
};

// The work of this workgroup: query head hq, prefilled query ins, tile.  The
// grid is one-dimensional over n_tiles x query heads, tile-major: all query
// heads of one tile are dealt before the next tile, and the tiles run from
// the longest (a query's last positions, which see the most keys; the queries
// are ordered by prompt length, longest first) to the shortest, so that the
// workgroups that start last are short.  Workgroups are dealt to the XCDs
// round-robin by index, and each XCD has its own L2; with xcd_map the heads
// are numbered so that all workgroups reading one kv-head's keys (a unit: its
// G query heads) run on the same XCD.
__device__ __forceinline__ void prefill_work(const PrefillArgs& a, int& hq, int32_t& ins,
                                             int32_t& tile) {
  const int32_t nq = a.n_attn / a.n_tiles;   // query heads
  const int32_t g = blockIdx.x / nq, j = blockIdx.x % nq;
  if (a.xcd_map) {
    const int32_t xcd = j % 8, k = j / 8;
    const int32_t u = xcd + 8 * (k / a.unit_heads);
    hq = u * a.unit_heads + k % a.unit_heads;
  } else {
    hq = j;
  }
  ins = 0;
  while (ins < a.n_ins - 1 && g >= a.tile_end[ins]) ++ins;
  tile = a.tile_end[ins] - 1 - g;   // the query's tiles, counted from its last one
}

// Appends prompt positions [t0, t0 + n) of kv-head h (threads tid of nthr).
template <int VPT>
__device__ __forceinline__ void prefill_append(const PrefillArgs& a, int b, int h, int32_t p,
                                               int64_t row0, int32_t t0, int32_t n, int tid,
                                               int nthr = kWave) {
  const int64_t ring_row = (int64_t)b * a.n_kv_heads + h;   // within the layer's rows
  u32x4* rk = reinterpret_cast<u32x4*>(a.k) + ring_row * a.cap * VPT;
  u32x4* rv = reinterpret_cast<u32x4*>(a.v) + ring_row * a.cap * VPT;
  const u32x4* kin = reinterpret_cast<const u32x4*>(a.knew);
  const u32x4* vin = reinterpret_cast<const u32x4*>(a.vnew);
  const int64_t c0 = a.base + a.L + a.T - p;   // < 2 * cap: base < cap, L + T <= cap
  for (int idx = tid; idx < n * VPT; idx += nthr) {
    const int32_t t = t0 + idx / VPT;
    const int e = idx % VPT;
    int64_t col = c0 + t;
    col = col >= a.cap ? col - a.cap : col;
    const int64_t src = ((row0 + t) * a.n_kv_heads + h) * VPT + e;
    rk[col * VPT + e] = kin[src];
    rv[col * VPT + e] = vin[src];
  }
}

// Any element type on the vector ALUs: a prompt position per lane group (LPT
// lanes, 16 bytes each), TPI positions per wave, the keys one at a time.
template <typename T, int D, int G>
__global__ void __launch_bounds__(kWave) prefill_valu_kernel(const PrefillArgs a) {
  using Geo = Geometry<T, D>;
  constexpr int EPL = Geo::kEpl, LPT = Geo::kLpt, TPI = Geo::kTpi, VPT = Geo::kVpt;
  const int lane = threadIdx.x;
  const int r = lane / LPT, cl = lane % LPT;
  int hq;
  int32_t ins, tile;
  prefill_work(a, hq, ins, tile);
  const int h = hq / G;
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

// bf16 on the matrix cores, flash-attention style: a workgroup of 4*S waves
// takes kPrefillTile prompt positions of one query head; four waves cover the
// positions (QG groups of 16 each) and S such quartets split the keys, each
// walking every S-th tile of KT keys (S tiles staged in LDS per iteration, K
// and V both as rows, 16-byte stores), and the quartets' softmax states merge
// through LDS at the end -- S shortens the longest causal tile's chain of
// iterations.  Every key and value fragment a wave reads from LDS serves its
// QG position groups: the kernel's limit is the LDS read bandwidth (each
// 32-key block costs a wave 16 KB of LDS reads, as many bytes as the matrix
// operations on one group take cycles), so QG = 2 halves the LDS bytes per
// multiply-add.
//  * QK^T: A = 16 key rows (lane l: key l % 16 of the half tile), B = 16 of
//    the wave's positions; the score of key 4*(l/16) + r (first 16 keys) and
//    16 + 4*(l/16) + r (next 16) for position l % 16 of the group lands in
//    lane l, register r.
//  * PV, transposed: O^T = V^T P^T.  B = P^T with k = 8*(l/16) + e standing
//    for key 4*(l/16) + e (e < 4) and 16 + 4*(l/16) + e - 4 (e >= 4) -- the
//    lane's own scores, in place; A = V^T in that key order, read with the
//    LDS transpose load (ds_read_b64_tr_b16): within a group of 16 lanes,
//    lane i receives element i % 4 of the 8-byte block addressed by lane
//    i / 4 + 4e, for e = 0..3; lane m of group g addresses key 4g + m / 4 at
//    columns 16*dt + 4*(m % 4), so lane i gets V[4g + e][16*dt + i].  Lane l
//    then holds output columns 16*dt + 4*(l/16) + r of position l % 16 of the
//    group: a position's rescale and normalisation stay in its own lanes, and
//    the max over the four lane groups uses the gfx950 row swaps.
//  * The weights' sum: one more operation per block, a column of ones as A
//    and the same P^T as B, so the sum is of the bf16 weights P·V was made
//    of, and every lane of a position holds it whole.
// Rows are padded to 8 dwords past a multiple of 32, so that the 16 rows of a
// transpose load spread over all banks.
// Keys per LDS tile and key stream: 32 (a stage of 64 keys with two streams,
// 37 KB of LDS) rather than 64, so that a workgroup's first stage arrives
// sooner and its last stage carries fewer keys past its diagonal.
#ifndef BATON_PREFILL_KT
#define BATON_PREFILL_KT 32
#endif
#ifndef BATON_PREFILL_LAZY
#define BATON_PREFILL_LAZY 8.0f
#endif
constexpr float kPrefillLazy = BATON_PREFILL_LAZY;
#ifndef BATON_PREFILL_QG
#define BATON_PREFILL_QG 1
#endif
constexpr int kPrefillGroups = BATON_PREFILL_QG;     // groups of 16 positions per wave
constexpr int kPrefillTile = 64 * kPrefillGroups;    // positions per workgroup

typedef short s16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ s16x4 lds_read_tr16(const uint8_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4*)(__attribute__((address_space(3))) void*)(p));
}

// Registers capped so that two workgroups share a CU (one group per wave: 128
// per lane, four waves per SIMD; two groups: 256, two waves per SIMD).
template <int D, int G, int S>
__global__ void __launch_bounds__(256 * S) __attribute__((amdgpu_waves_per_eu(kPrefillGroups == 1 ? 4 : 2)))
prefill_fa_kernel(const PrefillArgs a) {
  constexpr int VPT = D / 8, KK = D / 32, DT = D / 16;
  constexpr int QG = kPrefillGroups, TILE = kPrefillTile;
  constexpr int KT = BATON_PREFILL_KT;       // keys per LDS tile and key stream
  constexpr int ROW = D * 2 + 32;            // bytes per staged key / value row
  constexpr int NT = 256 * S;                // threads
  constexpr int NLD = KT * VPT / 256;        // 16-byte vectors per thread per stage, K and V each
  constexpr int GREC = DT * 4 + 2;           // floats of one group's softmax state per lane
  constexpr int REC = QG * GREC;
  static_assert((ROW / 4) % 32 == 8, "row padding");
  static_assert(S == 1 || (S - 1) * 4 * kWave * REC * 4 <= 2 * S * KT * ROW, "merge area");
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * S * KT * ROW];
  uint8_t* const ldsK = lds;
  uint8_t* const ldsV = lds + S * KT * ROW;
  const int tid = threadIdx.x;
  if ((int32_t)blockIdx.x >= a.n_attn) {
    // An append workgroup (after every attention workgroup in the grid, so
    // that these short ones fill the end of the launch): tile g of the
    // prefilled queries' prompt positions, kv-head h, into the ring.
    const int32_t j = (int32_t)blockIdx.x - a.n_attn;
    const int32_t g = j / a.n_kv_heads, h = j % a.n_kv_heads;
    int32_t ins = 0;
    while (ins < a.n_ins - 1 && g >= a.tile_end[ins]) ++ins;
    const int32_t tile = a.tile_end[ins] - 1 - g, p = a.plen[ins], b = a.slot[ins];
    const int64_t row0 = (int64_t)b * a.T + (a.T - p);
    prefill_append<VPT>(a, b, h, p, row0, tile * TILE, min(TILE, p - tile * TILE), tid, NT);
    return;
  }
  const int wave = tid / kWave, lane = tid % kWave;
  const int ks = wave / 4;                             // key stream of this wave
  const int g4 = lane / 16, c16 = lane % 16;
  int hq;
  int32_t ins, tile;
  prefill_work(a, hq, ins, tile);
  const int h = hq / G;
  const int b = a.slot[ins];
  const int32_t p = a.plen[ins];
  const int32_t wg0 = tile * TILE;                     // first position of the workgroup
  const int32_t i0 = wg0 + (wave % 4) * 16 * QG;       // first position of this wave
  const int64_t row0 = (int64_t)b * a.T + (a.T - p);
  const int nkv = a.n_kv_heads, nq = nkv * G;
  const u32x4* qin = reinterpret_cast<const u32x4*>(a.q);
  const u32x4* kin = reinterpret_cast<const u32x4*>(a.knew);
  const u32x4* vin = reinterpret_cast<const u32x4*>(a.vnew);
  const u32x4 zero = {0, 0, 0, 0};

  // A negative scale's sign is folded into q (negating a bf16 value is
  // exact), so that the softmax below always works with a positive factor:
  // the largest scaled score is then the scale times the largest score.
  const float qscale = fabsf(a.qscale);
  const uint32_t qsw = a.qscale < 0.f ? 0x80008000u : 0u;
  const u32x4 qsign = {qsw, qsw, qsw, qsw};
  bf16x8 qb[QG][KK];
#pragma unroll
  for (int gq = 0; gq < QG; ++gq) {
    const int32_t qi = i0 + 16 * gq + c16;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
      qb[gq][kk] = as_bf16x8(qi < p ? qin[((row0 + qi) * nq + hq) * VPT + kk * 4 + g4] ^ qsign : zero);
  }

  // Running max, the sums of the weights (ol: the weights as rounded to bf16
  // for the matrix operation, times a column of ones, on the matrix cores --
  // the output is then normalized by exactly the weights it was made of) and
  // the output accumulators.
  float m[QG], lsum[QG];
  f32x4 ol[QG];
  f32x4 o[QG][DT];
  const bf16x8 ones = __builtin_bit_cast(bf16x8, u32x4{0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u});
#pragma unroll
  for (int gq = 0; gq < QG; ++gq) {
    m[gq] = -INFINITY;
    ol[gq] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[gq][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  const int32_t wg_last = min(wg0 + TILE - 1, p - 1);
  // the wave's last position; a wave wholly past the prompt computes nothing
  const int32_t w_last = i0 < p ? min(i0 + 16 * QG - 1, p - 1) : -1;
  // This lane's transpose-load address within a value row block: key offset
  // 4*g4 + c16/4, columns 4*(c16 % 4).
  const int tr_off = (4 * g4 + c16 / 4) * ROW + (c16 % 4) * 8;
  // The prompt's keys and values of head h as raw buffers: token t's row at
  // byte t * nkv * D * 2; a token past the prompt gets an offset beyond the
  // range, which loads zeros (no branch, no wait per load).
  const uint32_t tok_bytes = (uint32_t)nkv * VPT * 16;
  const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<u32x4*>(kin + (row0 * nkv + h) * VPT), 0, (uint32_t)p * tok_bytes, kBufferWord3);
  const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<u32x4*>(vin + (row0 * nkv + h) * VPT), 0, (uint32_t)p * tok_bytes, kBufferWord3);
  u32x4 kr[NLD], vr[NLD];
  auto fetch = [&](int32_t kt, u32x4 (&kr)[NLD], u32x4 (&vr)[NLD]) {
#pragma unroll
    for (int u = 0; u < NLD; ++u) {
      const int v = tid + NT * u;
      const int32_t t = kt + v / VPT;
      const uint32_t off = t < p ? (uint32_t)t * tok_bytes + (uint32_t)(v % VPT) * 16u : 0x80000000u;
      kr[u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rk, off, 0, 0));
      vr[u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rv, off, 0, 0));
    }
  };
  auto compute = [&](int32_t k0) {
#pragma unroll
    for (int half = 0; half < KT / 32; ++half) {
      const int kb = ks * KT + 32 * half;              // key row of the block in the stage
      const int32_t tt = k0 + kb;
      if (tt > w_last) break;                          // wave-uniform
      f32x4 sa[QG], sb[QG];
#pragma unroll
      for (int gq = 0; gq < QG; ++gq) {
        sa[gq] = f32x4{0.f, 0.f, 0.f, 0.f};
        sb[gq] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const u32x4 ka = *reinterpret_cast<const u32x4*>(ldsK + (kb + c16) * ROW + (kk * 4 + g4) * 16);
        const u32x4 kc = *reinterpret_cast<const u32x4*>(ldsK + (kb + 16 + c16) * ROW + (kk * 4 + g4) * 16);
#pragma unroll
        for (int gq = 0; gq < QG; ++gq) {
          sa[gq] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ka), qb[gq][kk], sa[gq], 0, 0, 0);
          sb[gq] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kc), qb[gq][kk], sb[gq], 0, 0, 0);
        }
      }
      bf16x8 pa[QG];
#pragma unroll
      for (int gq = 0; gq < QG; ++gq) {
        const int32_t ig = i0 + 16 * gq;               // the group's first position
        const int32_t qi = ig + c16;
        // Unscaled scores; masked keys -inf.  A block whose 32 keys all come
        // before the group's first position is visible to every position of
        // the group and needs no mask (positions past the prompt are never
        // written).
        float s[8];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          s[r] = sa[gq][r];
          s[4 + r] = sb[gq][r];
        }
        if (tt + 31 > ig) {                            // wave-uniform
          const int32_t lim = qi < p ? qi - tt : -1;   // keys tt .. tt + lim are visible
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            s[r] = 4 * g4 + r <= lim ? s[r] : -INFINITY;
            s[4 + r] = 16 + 4 * g4 + r <= lim ? s[4 + r] : -INFINITY;
          }
        }
        float mx = s[0];
#pragma unroll
        for (int e = 1; e < 8; ++e) mx = fmaxf(mx, s[e]);
        mx = max_over_groups(mx) * qscale;             // qscale >= 0: the max of the scaled scores
        // The reference the weights are taken against moves only when the
        // block's maximum passes it by more than kPrefillLazy (base 2):
        // softmax does not depend on the reference, the weights stay below
        // 2^kPrefillLazy (well inside bf16's and fp32's range, at bf16's
        // relative precision), and the accumulators are rescaled -- this
        // lane's position by its own factor -- only when some position's
        // reference moved, which after the first keys is rare.
        if (__ballot(mx > m[gq] + kPrefillLazy)) {     // wave-uniform
          const float mn = mx > m[gq] + kPrefillLazy ? mx : m[gq];
          const float alpha = m[gq] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m[gq] - mn);
          ol[gq] *= alpha;
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) o[gq][dt] *= alpha;
          m[gq] = mn;
        }
        const float ref = m[gq] == -INFINITY ? 0.f : m[gq];
        // exponents are <= kPrefillLazy here: the hardware exp2 (results below
        // the smallest normal flush to 0, which a softmax weight may); the
        // scale is applied in the exponent's multiply-add
#pragma unroll
        for (int e = 0; e < 8; ++e) pa[gq][e] = (__bf16)__builtin_amdgcn_exp2f(fmaf(s[e], qscale, -ref));
      }
      const uint8_t* vblk = ldsV + kb * ROW + tr_off;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const s16x4 lo = lds_read_tr16(vblk + dt * 32);
        const s16x4 hi = lds_read_tr16(vblk + 16 * ROW + dt * 32);
        const s16x4 w2[2] = {lo, hi};
        const bf16x8 vb = __builtin_bit_cast(bf16x8, w2);
#pragma unroll
        for (int gq = 0; gq < QG; ++gq)
          o[gq][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vb, pa[gq], o[gq][dt], 0, 0, 0);
      }
#pragma unroll
      for (int gq = 0; gq < QG; ++gq) ol[gq] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pa[gq], ol[gq], 0, 0, 0);
    }
  };
  // The next stage's loads are in flight while the current one is computed.
  fetch(0, kr, vr);
  for (int32_t k0 = 0; k0 <= wg_last; k0 += S * KT) {   // bounds are workgroup-uniform
    __syncthreads();                                   // the previous stage is consumed
#pragma unroll
    for (int u = 0; u < NLD; ++u) {
      const int v = tid + NT * u;
      const int off = (v / VPT) * ROW + (v % VPT) * 16;
      *reinterpret_cast<u32x4*>(ldsK + off) = kr[u];
      *reinterpret_cast<u32x4*>(ldsV + off) = vr[u];
    }
    __syncthreads();
    if (k0 + S * KT <= wg_last) fetch(k0 + S * KT, kr, vr);
    compute(k0);
  }

  // Every lane of a position holds its whole sum (the operation summed over
  // the 32 keys of each block).
#pragma unroll
  for (int gq = 0; gq < QG; ++gq) lsum[gq] = ol[gq][0];
  if constexpr (S > 1) {
    // Key streams 1.. hand their states to stream 0 (same positions, same lane).
    __syncthreads();                                   // the stage buffers are free
    float* mrg = reinterpret_cast<float*>(lds) + ((ks - 1) * 4 + wave % 4) * kWave * REC + lane * REC;
    if (ks > 0) {
#pragma unroll
      for (int gq = 0; gq < QG; ++gq) {
        mrg[gq * GREC] = m[gq];
        mrg[gq * GREC + 1] = lsum[gq];
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int r = 0; r < 4; ++r) mrg[gq * GREC + 2 + dt * 4 + r] = o[gq][dt][r];
      }
    }
    __syncthreads();
    if (ks == 0) {
#pragma unroll
      for (int k = 1; k < S; ++k) {
        const float* src = reinterpret_cast<const float*>(lds) + ((k - 1) * 4 + wave % 4) * kWave * REC + lane * REC;
#pragma unroll
        for (int gq = 0; gq < QG; ++gq) {
          const float* sg = src + gq * GREC;
          const float m2 = sg[0];
          const float mm = fmaxf(m[gq], m2);
          const float fa = m[gq] == -INFINITY ? 0.f : exp2f(m[gq] - mm);
          const float fb = m2 == -INFINITY ? 0.f : exp2f(m2 - mm);
          lsum[gq] = lsum[gq] * fa + sg[1] * fb;
          m[gq] = mm;
#pragma unroll
          for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) o[gq][dt][r] = o[gq][dt][r] * fa + sg[2 + dt * 4 + r] * fb;
        }
      }
    }
  }
  if (ks == 0) {
    // Lane l holds columns 16 dt + 4 (l / 16) + r of position l % 16 of each group.
#pragma unroll
    for (int gq = 0; gq < QG; ++gq) {
      const int32_t qi = i0 + 16 * gq + c16;
      const float ls = lsum[gq];
      if (qi < p) {
        const float inv = 1.f / ls;
        uint16_t* o16 = reinterpret_cast<uint16_t*>(a.out) + ((row0 + qi) * nq + hq) * D + 4 * g4;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          *reinterpret_cast<uint2*>(o16 + 16 * dt) =
              make_uint2(f32_to_bf16_rne(o[gq][dt][0] * inv) | (f32_to_bf16_rne(o[gq][dt][1] * inv) << 16),
                         f32_to_bf16_rne(o[gq][dt][2] * inv) | (f32_to_bf16_rne(o[gq][dt][3] * inv) << 16));
      }
    }
  }
}

}  // namespace baton


