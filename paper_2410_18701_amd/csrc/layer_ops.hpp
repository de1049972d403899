// Kernels of a decode layer around the attention: the weight-streaming GEMM
// of the projections at decode batch sizes (up to 256 rows), RMS
// normalisation, the fused projection's split with rotary embedding of
// queries and keys, and the gated activation.  bf16 storage, fp32
// arithmetic, outputs rounded to nearest even.
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

// ------------------------------------------------------------ skinny GEMM --
// y[m][n] (+)= sum_k x[m][k] w[n][k] for m < rows <= 256: a linear layer at a
// decode step's batch.  The weight matrix (megabytes) is read once from HBM
// and dominates the traffic; x (rows x K) is small and stays in the caches.
// A workgroup takes up to 64 rows (MG <= 4 tiles of 16 per wave); past 64,
// the grid cuts the rows into chunks of 64 whose workgroups for one slice
// group run on the same XCD, so that the weight is read from HBM about once
// and from that XCD's L2 by the other chunks, and each wave takes two weight
// slices.  (Built as an alternative: all rows in one workgroup, MG = 8 or 16
// with shorter batches, KU = 2 or 1, so that the staged rows and their
// registers stay within bounds -- every weight block streamed once, but each
// read from LDS 16 times as often per block.)
//
// The weight is used in a packed form, made once per weight by
// pack_weight_kernel: 16-row slices of w, each a run of 1 KB blocks, one per
// step of 32 along k, block (s, t) holding at byte 16 l the eight elements
// w[16 s + l % 16][32 t + 8 (l / 16) ..] (zeros past N or K) -- exactly the A
// operand of v_mfma_f32_16x16x32_bf16 for lane l.  A wave owns one slice (four
// per workgroup) and streams its blocks with one contiguous 1 KB load per
// step, so every weight row is read in long bursts (in the stored row-major
// layout a wave would touch 16 rows 64 bytes at a time, which the DRAM serves
// at a fraction of its bandwidth).  When there are too few slices to occupy
// the GPU the steps are also split into S ranges whose fp32 partial sums
// gemm_reduce_kernel adds up.  x's rows are the B operand, 16 at a time (lane
// l: row 16 j + l % 16, the same k group); lane l then holds outputs
// (n0 + 4 (l / 16) + r, 16 j + l % 16), r < 4.  Loads are raw buffer loads
// whose out-of-range offsets return zeros: x rows past `rows` and k past K
// need no branch.
typedef __bf16 gemm_bf16x8 __attribute__((ext_vector_type(8)));
typedef float gemm_f32x4 __attribute__((ext_vector_type(4)));

struct SkinnyArgs {
  const uint16_t* x;     // [rows][K]
  const uint16_t* wp;    // packed weight: [ceil(N / 16)][ceil(K / 32)] blocks of 512 elements
  uint16_t* y;           // [rows][N]
  float* part;           // [S][rows][N] fp32, when S > 1
  int32_t rows, N, K;    // rows <= 256
  int32_t chunks;        // row chunks: ceil(rows / 64), or 1
  int32_t groups;        // slice groups (workgroups per chunk)
  int32_t kt;            // blocks per slice, ceil(K / 32)
  int32_t tc;            // blocks per split
  int32_t accumulate;    // 1: y += x . w^T
  int32_t gated;         // F > 0: w is [gate; up] (2F rows), y [rows][F] = silu(x . gate^T) * (x . up^T)
};

#ifndef BATON_GEMM_WAVES
#define BATON_GEMM_WAVES 4
#endif
constexpr int32_t kGemmWaves = BATON_GEMM_WAVES;   // weight slices per workgroup
constexpr uint32_t kGemmOob = 0x80000000u;   // an offset past every buffer's range
constexpr int32_t kGemmBufWord3 = 0x00020000;

template <int AUX>   // 2: non-temporal
__device__ __forceinline__ u32x4 gemm_load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, AUX));
}

// One thread per 16-byte piece of the packed weight.
__global__ void __launch_bounds__(256) pack_weight_kernel(const u32x4* __restrict__ w, u32x4* __restrict__ wp,
                                                          int32_t N, int32_t K, int32_t kt, int64_t n_pieces) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n_pieces) return;
  const int32_t l = (int32_t)(i % kWave);
  const int64_t blk = i / kWave;
  const int32_t t = (int32_t)(blk % kt);
  const int32_t n = (int32_t)(blk / kt) * 16 + l % 16, k = 32 * t + 8 * (l / 16);
  wp[i] = (n < N && k < K) ? w[((int64_t)n * K + k) / 8] : u32x4{0, 0, 0, 0};
}

// Activation rows staged in LDS per batch of KU blocks: the workgroup's rows
// (64, or 16 MG past 64) of 64 KU bytes, each padded by 16 bytes so that the
// 16 rows one B-operand read spans fall in different banks.
template <int KU, int MG>
struct GemmLds {
  static constexpr int kRows = 16 * MG > 64 ? 16 * MG : 64;   // rows of x per workgroup
  static constexpr int kRow = 64 * KU + 16;   // bytes per staged row
  static constexpr int kBuf = kRows * kRow;   // one batch of the rows
  static constexpr int kPieces = 4 * KU;      // 16-byte pieces per row and batch
};

// The (slice group, row chunk) of a workgroup.  One chunk: the group is the
// workgroup index.  Several: workgroups are dealt to the GPU's eight XCDs in
// turn (index mod 8), so the chunks of one group go to indices 8 apart -- the
// same XCD, dispatched one after the other -- and the weight blocks they all
// read come from that XCD's L2 after the first read; the grid is padded to
// whole sets of 8 groups, the padding workgroups doing nothing.
__device__ __forceinline__ bool gemm_tile(const SkinnyArgs& a, int32_t& grp, int32_t& chunk) {
  if (a.chunks == 1) {
    grp = (int32_t)blockIdx.x;
    chunk = 0;
    return true;
  }
  const int32_t b = (int32_t)blockIdx.x, j = b / 8;
  chunk = j % a.chunks;
  grp = (j / a.chunks) * 8 + b % 8;
  return grp < a.groups;
}

// WAUX: the weight loads' cache policy, 2 (non-temporal) when each weight
// block is read once (one row chunk), 0 when the group's other chunks read it
// again from L2.  P: register sets of the load pipeline.  NS: weight slices
// per wave; with NS > 1 every activation
// operand a wave reads from LDS feeds NS matrix operations instead of one,
// which matters past 64 rows, where the workgroup's LDS reads would otherwise
// take as long as its matrix operations.
template <int MG, int KU, int WAUX, int NS, int P>
__global__ void __launch_bounds__(kWave * kGemmWaves) skinny_gemm_kernel(const SkinnyArgs a) {
  using Lds = GemmLds<KU, MG>;
  constexpr int kXPer = Lds::kRows * Lds::kPieces / (kWave * kGemmWaves);   // activation pieces per thread and batch
  static_assert(NS * MG * 2 * kWave * 8 <= 2 * Lds::kBuf, "gated exchange area: both staging buffers");
  __shared__ __attribute__((aligned(16))) uint8_t xs[2][Lds::kBuf];
  const int tid = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int lane = tid % kWave, c16 = lane % 16, g4 = lane / 16;
  // Gated: waves 0 and 1 take gate slices 2 NS x + NS w + i, waves 2 and 3 the
  // up slices of the same output columns (F / 16 further).
  static_assert(kGemmWaves == 4, "the gated epilogue pairs two gate and two up waves");
  int32_t grp, chunk;   // slice group, and the workgroup's rows of x and y
  if (!gemm_tile(a, grp, chunk)) return;   // the whole workgroup: padding
  const int32_t slice0 = a.gated ? (w < 2 ? 2 * NS * grp + NS * w : a.gated / 16 + 2 * NS * grp + NS * (w - 2))
                                 : (grp * kGemmWaves + w) * NS;
  const int32_t t_begin = blockIdx.y * a.tc, t_end = min(a.kt, t_begin + a.tc);
  const uint32_t row_bytes = (uint32_t)a.K * 2u;
  __amdgpu_buffer_rsrc_t rw[NS];   // slice i: empty past N (loads zeros, writes nothing)
#pragma unroll
  for (int i = 0; i < NS; ++i) {
    const int32_t slice = slice0 + i;
    rw[i] = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(a.wp) + ((int64_t)min(slice, (a.N + 15) / 16) * a.kt + t_begin) * 512, 0,
        16 * slice < a.N ? (t_end - t_begin) * 1024 : 0, kGemmBufWord3);
  }
  const int32_t xrow0 = Lds::kRows * chunk, rows = min(Lds::kRows, a.rows - xrow0);
  const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.x) + (int64_t)xrow0 * a.K, 0, (int32_t)(rows * row_bytes), kGemmBufWord3);

  gemm_f32x4 acc[NS][MG];
#pragma unroll
  for (int i = 0; i < NS; ++i)
#pragma unroll
    for (int j = 0; j < MG; ++j) acc[i][j] = gemm_f32x4{0.f, 0.f, 0.f, 0.f};

  // Loads of batch b (blocks t_begin + KU b ...): the workgroup's activation
  // pieces (thread tid: pieces tid + 64 kGemmWaves i -- row p / (4 KU), 16 bytes at
  // 16 (p % (4 KU)) of the batch) and this wave's weight blocks, both issued
  // unconditionally (past the end they return zeros).
  auto issue = [&](int32_t b, u32x4 (&xr)[kXPer], u32x4 (&wr)[NS][KU]) {
    const int32_t tb = t_begin + KU * b;
#pragma unroll
    for (int i = 0; i < kXPer; ++i) {
      const int32_t p = tid + kWave * kGemmWaves * i;
      const int32_t m = p / Lds::kPieces, c = p % Lds::kPieces;
      const int32_t k = 32 * tb + 8 * c;
      xr[i] = gemm_load<0>(rx, (m < rows && k < a.K && tb + c / 4 < t_end)
                                   ? (uint32_t)m * row_bytes + (uint32_t)k * 2u : kGemmOob);
    }
#pragma unroll
    for (int u = 0; u < KU; ++u) {
      const uint32_t off = tb + u < t_end ? (uint32_t)(tb + u - t_begin) * 1024u + (uint32_t)lane * 16u : kGemmOob;
#pragma unroll
      for (int i = 0; i < NS; ++i) wr[i][u] = gemm_load<WAUX>(rw[i], off);
    }
  };
  auto stage = [&](int buf, const u32x4 (&xr)[kXPer]) {
#pragma unroll
    for (int i = 0; i < kXPer; ++i) {
      const int32_t p = tid + kWave * kGemmWaves * i;
      *reinterpret_cast<u32x4*>(&xs[buf][(p / Lds::kPieces) * Lds::kRow + (p % Lds::kPieces) * 16]) = xr[i];
    }
  };
  auto mult = [&](int buf, const u32x4 (&wr)[NS][KU]) {
#pragma unroll
    for (int u = 0; u < KU; ++u) {
      u32x4 xb[MG];
#pragma unroll
      for (int j = 0; j < MG; ++j)
        xb[j] = *reinterpret_cast<const u32x4*>(&xs[buf][(16 * j + c16) * Lds::kRow + (32 * u + 8 * g4) * 2]);
#pragma unroll
      for (int j = 0; j < MG; ++j)
#pragma unroll
        for (int i = 0; i < NS; ++i)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(gemm_bf16x8, wr[i][u]),
                                                              __builtin_bit_cast(gemm_bf16x8, xb[j]), acc[i][j], 0,
                                                              0, 0);
    }
  };
  // P register sets: while batch b is multiplied, batches b + 1 .. b + P - 1
  // are in flight (every batch's activation loads are issued ahead of its
  // weight loads, so waiting for activations never waits for weights), and
  // batch b + 1's activations, issued P - 2 batches earlier, go to LDS at the
  // end of the step.  Batch b's activations are in LDS buffer b & 1.  Sets are
  // indexed by constants only (the steps are unrolled), so they stay in
  // registers.
  const int32_t n_batch = (t_end - t_begin + KU - 1) / KU;   // the same for the whole workgroup
  if (n_batch > 0) {
    u32x4 xr[P][kXPer], wr[P][NS][KU];
#pragma unroll
    for (int q = 0; q < P - 1; ++q) issue(q, xr[q], wr[q]);
    stage(0, xr[0]);
    __syncthreads();
#define BATON_GEMM_STEP(S)                                               \
  issue(b + (S) + P - 1, xr[((S) + P - 1) % P], wr[((S) + P - 1) % P]); \
  __builtin_amdgcn_sched_barrier(0);                                     \
  mult((b + (S)) & 1, wr[(S) % P]);                                      \
  stage((b + (S) + 1) & 1, xr[((S) + 1) % P]);                           \
  __syncthreads();
    // A counted loop with no exit inside its body (an exit between the steps
    // makes the compiler drain every load in flight at the loop head), then
    // the last n_batch % P steps.
    int32_t b = 0;
    for (; b + P <= n_batch; b += P) {
#pragma unroll
      for (int q = 0; q < P; ++q) {
        BATON_GEMM_STEP(q)
      }
    }
#pragma unroll
    for (int q = 0; q < P - 1; ++q) {
      if (b + q >= n_batch) break;
      BATON_GEMM_STEP(q)
    }
#undef BATON_GEMM_STEP
  }
  if (a.gated) {
    // The up waves hand their outputs, rounded to bf16 as the product's output
    // would be, to the gate waves through LDS (free: the loop ended on a
    // barrier, after which neither staging buffer is read again); lane l of
    // both holds the same (row, column).  The activation
    // is then silu_mul_kernel's arithmetic on the rounded values.
    uint2* ex = reinterpret_cast<uint2*>(&xs[0][0]);   // [2 waves][NS][MG][64 lanes]
    if (w >= 2) {
#pragma unroll
      for (int i = 0; i < NS; ++i)
#pragma unroll
        for (int j = 0; j < MG; ++j)
          ex[(((w - 2) * NS + i) * MG + j) * kWave + lane] =
              make_uint2(pack_bf16(acc[i][j][0], acc[i][j][1]), pack_bf16(acc[i][j][2], acc[i][j][3]));
    }
    __syncthreads();
    if (w < 2) {
#pragma unroll
      for (int i = 0; i < NS; ++i) {
        const int32_t n = 16 * (slice0 + i) + 4 * g4;
        if (n >= a.gated) continue;
#pragma unroll
        for (int j = 0; j < MG; ++j) {
          const int32_t m = 16 * j + c16;
          if (m >= rows) continue;
          const uint2 u = ex[((w * NS + i) * MG + j) * kWave + lane];
          const uint32_t gw[2] = {pack_bf16(acc[i][j][0], acc[i][j][1]), pack_bf16(acc[i][j][2], acc[i][j][3])};
          const uint32_t uw[2] = {u.x, u.y};
          uint32_t o[2];
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            const float g0 = bf16_lo(gw[q]), g1 = bf16_hi(gw[q]);
            const float s0 = g0 / (1.f + expf(-g0)), s1 = g1 / (1.f + expf(-g1));
            o[q] = pack_bf16(s0 * bf16_lo(uw[q]), s1 * bf16_hi(uw[q]));
          }
          *reinterpret_cast<uint2*>(a.y + (int64_t)(xrow0 + m) * a.gated + n) = make_uint2(o[0], o[1]);
        }
      }
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < NS; ++i) {
    const int32_t n = 16 * (slice0 + i) + 4 * g4;
    if (n >= a.N) continue;
#pragma unroll
    for (int j = 0; j < MG; ++j) {
      const int32_t m = 16 * j + c16;
      if (m >= rows) continue;
      if (gridDim.y > 1) {
        *reinterpret_cast<float4*>(a.part + ((int64_t)blockIdx.y * a.rows + xrow0 + m) * a.N + n) =
            make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
      } else {
        uint2* yp = reinterpret_cast<uint2*>(a.y + (int64_t)(xrow0 + m) * a.N + n);
        float v0 = acc[i][j][0], v1 = acc[i][j][1], v2 = acc[i][j][2], v3 = acc[i][j][3];
        if (a.accumulate) {
          const uint2 old = *yp;
          v0 += bf16_lo(old.x); v1 += bf16_hi(old.x); v2 += bf16_lo(old.y); v3 += bf16_hi(old.y);
        }
        *yp = make_uint2(pack_bf16(v0, v1), pack_bf16(v2, v3));
      }
    }
  }
}

// y[m][n] (+)= sum over the S splits of part[s][m][n], 4 outputs per thread,
// the splits added in order.
__global__ void __launch_bounds__(256) gemm_reduce_kernel(const float* __restrict__ part, uint16_t* __restrict__ y,
                                                          int32_t S, int64_t n_out, int32_t accumulate) {
  const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (i >= n_out) return;
  float4 v = *reinterpret_cast<const float4*>(part + i);
  for (int32_t s = 1; s < S; ++s) {
    const float4 p = *reinterpret_cast<const float4*>(part + s * n_out + i);
    v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
  }
  uint2* yp = reinterpret_cast<uint2*>(y + i);
  if (accumulate) {
    const uint2 old = *yp;
    v.x += bf16_lo(old.x); v.y += bf16_hi(old.x); v.z += bf16_lo(old.y); v.w += bf16_hi(old.y);
  }
  *yp = make_uint2(pack_bf16(v.x, v.y), pack_bf16(v.z, v.w));
}

// The split sums of a projection's output added up (and to the residual y
// with accumulate) as gemm_reduce_kernel does, then each row's RMS norm as
// rmsnorm_kernel does, element for element and in the same order: one
// workgroup per row, thread t owning the row's 8-element groups t, t +
// kRowThreads, ...  The result is bit-identical to the two launches, without
// the second one's read of y.
__global__ void __launch_bounds__(kRowThreads) reduce_rmsnorm_kernel(
    const float* __restrict__ part, uint16_t* __restrict__ y, int32_t S, int64_t n_out, int32_t accumulate,
    const u32x4* __restrict__ g, u32x4* __restrict__ yn, int32_t vec_per_row, float inv_dim, float eps) {
  __shared__ float psum[kRowThreads / kWave];
  const int64_t row = blockIdx.x;
  u32x4* yr = reinterpret_cast<u32x4*>(y) + row * vec_per_row;
  float ss = 0.f;
  for (int i = threadIdx.x; i < vec_per_row; i += kRowThreads) {
    const int64_t e0 = (row * vec_per_row + i) * 8;   // the group's first element
    const u32x4 old = accumulate ? yr[i] : u32x4{0, 0, 0, 0};
    u32x4 w;
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      float4 v = *reinterpret_cast<const float4*>(part + e0 + 4 * hf);
      for (int32_t s = 1; s < S; ++s) {
        const float4 q = *reinterpret_cast<const float4*>(part + s * n_out + e0 + 4 * hf);
        v.x += q.x; v.y += q.y; v.z += q.z; v.w += q.w;
      }
      if (accumulate) {
        v.x += bf16_lo(old[2 * hf]); v.y += bf16_hi(old[2 * hf]);
        v.z += bf16_lo(old[2 * hf + 1]); v.w += bf16_hi(old[2 * hf + 1]);
      }
      w[2 * hf] = pack_bf16(v.x, v.y);
      w[2 * hf + 1] = pack_bf16(v.z, v.w);
    }
    yr[i] = w;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float a = bf16_lo(w[j]), b = bf16_hi(w[j]);
      ss = fmaf(a, a, fmaf(b, b, ss));
    }
  }
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) ss += __shfl_xor(ss, off, kWave);
  if (threadIdx.x % kWave == 0) psum[threadIdx.x / kWave] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kRowThreads / kWave; ++w) tot += psum[w];
  const float inv = 1.0f / sqrtf(tot * inv_dim + eps);
  for (int i = threadIdx.x; i < vec_per_row; i += kRowThreads) {
    const u32x4 w = yr[i], gw = g[i];   // this thread's own stores above
    u32x4 o;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      o[j] = pack_bf16(bf16_lo(w[j]) * inv * bf16_lo(gw[j]), bf16_hi(w[j]) * inv * bf16_hi(gw[j]));
    yn[row * vec_per_row + i] = o;
  }
}

}  // namespace
}  // namespace baton
