// Elementwise and row kernels of a decode layer around the attention (the
// GEMMs are hipBLASLt's): RMS normalisation, the fused projection's split with
// rotary embedding of queries and keys, and the gated activation.  bf16
// storage, fp32 arithmetic, outputs rounded to nearest even.
#pragma once

#include "common.hpp"

namespace baton {
namespace {   // internal linkage: the kernels are included by two translation units

constexpr int kRowThreads = 256;

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  return f32_to_bf16_rne(lo) | (f32_to_bf16_rne(hi) << 16);
}

// y[r] = x[r] / sqrt(mean(x[r]^2) + eps) * g, one workgroup per row; dim a
// multiple of 8 (16-byte vectors).
__global__ void __launch_bounds__(kRowThreads) rmsnorm_kernel(const u32x4* __restrict__ x,
                                                              const u32x4* __restrict__ g,
                                                              u32x4* __restrict__ y, int32_t vec_per_row,
                                                              float inv_dim, float eps) {
  __shared__ float part[kRowThreads / kWave];
  const int64_t row = blockIdx.x;
  const u32x4* xr = x + row * vec_per_row;
  float ss = 0.f;
  for (int i = threadIdx.x; i < vec_per_row; i += kRowThreads) {
    const u32x4 w = xr[i];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float a = bf16_lo(w[j]), b = bf16_hi(w[j]);
      ss = fmaf(a, a, fmaf(b, b, ss));
    }
  }
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) ss += __shfl_xor(ss, off, kWave);
  if (threadIdx.x % kWave == 0) part[threadIdx.x / kWave] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kRowThreads / kWave; ++w) tot += part[w];
  const float inv = 1.0f / sqrtf(tot * inv_dim + eps);
  for (int i = threadIdx.x; i < vec_per_row; i += kRowThreads) {
    const u32x4 w = xr[i], gw = g[i];
    u32x4 o;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      o[j] = pack_bf16(bf16_lo(w[j]) * inv * bf16_lo(gw[j]), bf16_hi(w[j]) * inv * bf16_hi(gw[j]));
    y[row * vec_per_row + i] = o;
  }
}

// Split of the fused projection qkv [B][(Hq + 2 Hkv) D] into q [B][Hq][D],
// k [B][Hkv][D] (both rotated) and v [B][Hkv][D].  One wave per (row, head):
// lane i < D/2 rotates pair (i, i + D/2) by pos_b * theta^(-2i/D).  The angle
// is formed and reduced modulo 2 pi in double precision, its sine and cosine
// then taken in single precision on [-pi, pi].
struct RopeArgs {
  const uint16_t* qkv;
  uint16_t* q;
  uint16_t* k;
  uint16_t* v;
  int32_t n_q_heads, n_kv_heads, head_dim;
  double log2_theta;
  int32_t pos[512];
};

__global__ void __launch_bounds__(kWave) rope_qkv_kernel(const RopeArgs a) {
  const int hq = a.n_q_heads, hkv = a.n_kv_heads, D = a.head_dim, half = D / 2;
  const int heads = hq + 2 * hkv;
  const int b = blockIdx.x / heads, head = blockIdx.x - b * heads;
  const uint16_t* src = a.qkv + ((int64_t)b * heads + head) * D;
  const int i = threadIdx.x;
  if (head >= hq + hkv) {                      // a value head: copied
    uint16_t* dst = a.v + ((int64_t)b * hkv + (head - hq - hkv)) * D;
    for (int e = i; e < D; e += kWave) dst[e] = src[e];
    return;
  }
  if (i >= half) return;
  const double inv = exp2(-(double)(2 * i) / D * a.log2_theta);
  const double two_pi = 6.283185307179586;
  double ang = (double)a.pos[b] * inv;
  ang -= two_pi * rint(ang / two_pi);
  float s, c;
  sincosf((float)ang, &s, &c);
  const float x0 = __uint_as_float((uint32_t)src[i] << 16);
  const float x1 = __uint_as_float((uint32_t)src[i + half] << 16);
  uint16_t* dst = head < hq ? a.q + ((int64_t)b * hq + head) * D : a.k + ((int64_t)b * hkv + (head - hq)) * D;
  dst[i] = (uint16_t)f32_to_bf16_rne(x0 * c - x1 * s);
  dst[i + half] = (uint16_t)f32_to_bf16_rne(x0 * s + x1 * c);
}

// out[r][j] = silu(gate_up[r][j]) * gate_up[r][F + j], 8 elements per thread.
__global__ void __launch_bounds__(256) silu_mul_kernel(const u32x4* __restrict__ gu, u32x4* __restrict__ out,
                                                       int32_t vec_per_row, int64_t n_vec) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n_vec) return;
  const int64_t r = i / vec_per_row, c = i - r * vec_per_row;
  const u32x4 g = gu[r * 2 * vec_per_row + c], u = gu[r * 2 * vec_per_row + vec_per_row + c];
  u32x4 o;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float g0 = bf16_lo(g[j]), g1 = bf16_hi(g[j]);
    const float s0 = g0 / (1.f + expf(-g0)), s1 = g1 / (1.f + expf(-g1));
    o[j] = pack_bf16(s0 * bf16_lo(u[j]), s1 * bf16_hi(u[j]));
  }
  out[i] = o;
}

}  // namespace
}  // namespace baton
