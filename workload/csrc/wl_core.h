/*
 * Seeded, counter-based value generator for synthetic decode workloads.
 *
 * This header holds input generation only: no step of the re-batching method.
 * It is compiled twice, once by gcc for the host library and once by hipcc for
 * the device library, so that a tensor filled on the GPU and the same tensor
 * filled on the host carry identical bits.  Define WL_QUAL before including it
 * to give the functions the qualifiers of the compiling side.
 *
 * Bit source: SplitMix64 (G. Steele, D. Lea, C. Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014), used in counter mode: the
 * j-th output of a stream with key k is mix64(k + (j + 1) * gamma).  mix64 is
 * the published SplitMix64 output function (Stafford's "Mix13" constants).
 *
 * Value: an Irwin-Hall sum of twelve 16-bit uniforms, centred.  With k_i
 * uniform on {0..65535}, x = (2 * sum k_i - 12 * 65535) * 2^-17 has mean 0 and
 * variance (4 * 12 * (65536^2 - 1) / 12) * 2^-34 = 1 - 2^-32, |x| < 6, and is
 * an integer times 2^-17 with |integer| < 2^20: exactly representable in fp32,
 * so no rounding (and no libm call) enters the value on either side.
 * bf16 storage rounds that fp32 to nearest-even with integer operations.
 */
#ifndef BATON_WL_CORE_H
#define BATON_WL_CORE_H

#include <stdint.h>

#ifndef WL_QUAL
#define WL_QUAL static inline
#endif

#define WL_GAMMA 0x9E3779B97F4A7C15ull

WL_QUAL uint64_t wl_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

/* Key of stream `stream` under `seed`. */
WL_QUAL uint64_t wl_stream_key(uint64_t seed, uint64_t stream) {
  return wl_mix64(seed * WL_GAMMA + stream);
}

/* j-th 64-bit output (j >= 0) of the stream with key `key`. */
WL_QUAL uint64_t wl_draw(uint64_t key, uint64_t j) {
  return wl_mix64(key + (j + 1ull) * WL_GAMMA);
}

WL_QUAL int32_t wl_sum16x4(uint64_t w) {
  return (int32_t)(w & 0xFFFFull) + (int32_t)((w >> 16) & 0xFFFFull) +
         (int32_t)((w >> 32) & 0xFFFFull) + (int32_t)(w >> 48);
}

/* Approximately N(0,1) value of element counter c: draws 3c, 3c+1, 3c+2. */
WL_QUAL float wl_normal(uint64_t key, uint64_t c) {
  const uint64_t j = 3ull * c;
  const int32_t s = wl_sum16x4(wl_draw(key, j)) + wl_sum16x4(wl_draw(key, j + 1)) +
                    wl_sum16x4(wl_draw(key, j + 2));
  const int32_t t = 2 * s - 12 * 65535;
  return (float)t * (1.0f / 131072.0f);
}

WL_QUAL uint32_t wl_f32_bits(float f) {
  union { float f; uint32_t u; } x;
  x.f = f;
  return x.u;
}

/* fp32 -> bf16 round to nearest even (inputs here are finite). */
WL_QUAL uint16_t wl_bf16_rne(float f) {
  const uint32_t u = wl_f32_bits(f);
  const uint32_t r = u + 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(r >> 16);
}

/* Element codes of the fill routines. */
#define WL_F32 0
#define WL_BF16 1

#endif
