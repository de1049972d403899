// Device helpers shared by the baton kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace baton {

constexpr int kWave = 64;

// 16 bytes per lane: the widest global load/store of one lane.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Storage traits: fp32 or bf16 elements, handled as raw bits.
struct F32Tag {
  static constexpr int kBytes = 4;
};
struct BF16Tag {
  static constexpr int kBytes = 2;
};

__device__ __forceinline__ float bits_to_f32(uint32_t u) { return __uint_as_float(u); }

// The two bf16 halves of a 32-bit word, widened exactly to fp32.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// fp32 -> bf16 bits, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (u >> 16) | 0x0040u;
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Widen the elements one lane holds in 16 bytes: 4 fp32 or 8 bf16.
template <typename T>
struct Lane16;

template <>
struct Lane16<F32Tag> {
  static constexpr int kElems = 4;
  __device__ __forceinline__ static void widen(const u32x4& w, float* x) {
    x[0] = bits_to_f32(w.x);
    x[1] = bits_to_f32(w.y);
    x[2] = bits_to_f32(w.z);
    x[3] = bits_to_f32(w.w);
  }
  __device__ __forceinline__ static u32x4 narrow(const float* x) {
    u32x4 w;
    w.x = __float_as_uint(x[0]);
    w.y = __float_as_uint(x[1]);
    w.z = __float_as_uint(x[2]);
    w.w = __float_as_uint(x[3]);
    return w;
  }
};

template <>
struct Lane16<BF16Tag> {
  static constexpr int kElems = 8;
  __device__ __forceinline__ static void widen(const u32x4& w, float* x) {
    x[0] = bf16_lo(w.x);
    x[1] = bf16_hi(w.x);
    x[2] = bf16_lo(w.y);
    x[3] = bf16_hi(w.y);
    x[4] = bf16_lo(w.z);
    x[5] = bf16_hi(w.z);
    x[6] = bf16_lo(w.w);
    x[7] = bf16_hi(w.w);
  }
  __device__ __forceinline__ static u32x4 narrow(const float* x) {
    u32x4 w;
    w.x = f32_to_bf16_rne(x[0]) | (f32_to_bf16_rne(x[1]) << 16);
    w.y = f32_to_bf16_rne(x[2]) | (f32_to_bf16_rne(x[3]) << 16);
    w.z = f32_to_bf16_rne(x[4]) | (f32_to_bf16_rne(x[5]) << 16);
    w.w = f32_to_bf16_rne(x[6]) | (f32_to_bf16_rne(x[7]) << 16);
    return w;
  }
};

// Base-2 exponential by the hardware instruction alone (no range fix-up):
// results below 2^-126 flush to zero, which leaves a softmax sum -- whose
// largest term is 1 -- unchanged in fp32; exp2(-inf) = 0.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Cross-lane moves inside a row of 16 lanes (DPP), for reductions over the
// lanes that share one token row.
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, true));
}
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // lane i <-> 7 - i within each 8
constexpr int kDppMirror = 0x140;     // lane i <-> 15 - i within each 16

// Sum over aligned groups of N consecutive lanes (N in {4, 8, 16, 32}); every
// lane of a group receives the group's sum.  Must run with all lanes active.
template <int N>
__device__ __forceinline__ float group_sum(float x) {
  static_assert(N == 4 || N == 8 || N == 16 || N == 32, "group size");
  x += dpp<kDppXor1>(x);
  x += dpp<kDppXor2>(x);
  if constexpr (N >= 8) x += dpp<kDppHalfMirror>(x);
  if constexpr (N >= 16) x += dpp<kDppMirror>(x);
  if constexpr (N >= 32) x += __shfl_xor(x, 16, kWave);
  return x;
}

// Reductions over the four lane groups of 16 (lanes l, l ^ 16, l ^ 32, l ^ 48)
// with the gfx950 row swaps: each swap hands every lane its own value and its
// partner's, without a trip through LDS.
__device__ __forceinline__ float max_over_groups(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const uint32_t v = __float_as_uint(x);
  const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float sum_over_groups(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const uint32_t v = __float_as_uint(x);
  const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Ring column arithmetic: a + b mod cap for 0 <= a, b < cap.
__device__ __forceinline__ int64_t ring_add(int64_t a, int64_t b, int64_t cap) {
  const int64_t s = a + b;
  return s >= cap ? s - cap : s;
}

constexpr int kMaxHoles = 64;       // == BATON_MAX_HOLES

// Holes of live rows: the padding columns a prefill step inside the batch
// leaves behind the latest token of the other rows.  Hole k covers the
// logical columns [col0[k], col1[k]); holes are sorted by column, and a row's
// holes are a suffix of the list, from index first[b].
struct HoleList {
  int32_t n;
  int32_t col[kMaxHoles][2];
};

// Calls f(t0, t1) for each run of consecutive tokens of a live row with n
// cached tokens (token t is logical column L - n + t; token n is the current
// one): [0, n + 1) without the row's holes.
template <typename F>
__host__ __device__ __forceinline__ void row_runs(const HoleList& hl, int32_t first, int64_t L,
                                                  int32_t n, F&& f) {
  const int32_t c0 = (int32_t)(L - n);   // logical columns fit int32 (the hole list holds them so)
  int32_t t = 0;
  const int kn = hl.n;
  // the next hole is read while the current one is handled
  int32_t a0 = first < kn ? hl.col[first][0] : 0, a1 = first < kn ? hl.col[first][1] : 0;
  for (int k = first; k < kn; ++k) {
    const int32_t h0 = a0 - c0, h1 = a1 - c0;
    if (k + 1 < kn) {
      a0 = hl.col[k + 1][0];
      a1 = hl.col[k + 1][1];
    }
    if (h1 <= 0 || h0 > n) continue;   // outside the row (never for a row's own holes)
    if (h0 > t) f(t, h0);
    t = h1 > t ? h1 : t;
  }
  if (t < n + 1) f(t, n + 1);
}

}  // namespace baton
