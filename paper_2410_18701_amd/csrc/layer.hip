// Host side of the decode-layer operations around the attention: the
// projections on the library's weight-streaming GEMM over packed weights (up
// to 256 rows), launches of the row and elementwise kernels.
// The C ABI is documented in include/baton.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <new>

#include "baton.h"
#include "layer_ops.hpp"

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#ifndef BATON_GEMM_TARGET_WAVES
#define BATON_GEMM_TARGET_WAVES 1024   // weight slices x splits when the slices alone are too few
#endif
#ifndef BATON_GEMM_MIN_SLICES
#define BATON_GEMM_MIN_SLICES 512      // from this many slices on, no split along k
#endif
#ifndef BATON_GEMM_KU
#define BATON_GEMM_KU 4                // 1 KB weight blocks per load batch of a wave
#endif
#ifndef BATON_GEMM_MIN_WAVES_WIDE
#define BATON_GEMM_MIN_WAVES_WIDE 768  // past 64 rows: from this many waves on, no split along k
#endif
#ifndef BATON_GEMM_TARGET_WAVES_WIDE
#define BATON_GEMM_TARGET_WAVES_WIDE 1024
#endif

#ifndef BATON_GEMM_WIDE
#define BATON_GEMM_WIDE 0              // past 64 rows: 1: all rows per workgroup; 0: chunks of 64 rows
#endif

#ifndef BATON_GEMM_NS_WIDE
#define BATON_GEMM_NS_WIDE 2           // past 64 rows: weight slices per wave
#endif
#ifndef BATON_GEMM_KU_WIDE
#define BATON_GEMM_KU_WIDE 2           // past 64 rows: 1 KB weight blocks per slice and load batch
#endif
#ifndef BATON_GEMM_MG_WIDE
#define BATON_GEMM_MG_WIDE 4           // past 64 rows: row tiles of 16 per chunk
#endif

#ifndef BATON_GEMM_DEPTH
#define BATON_GEMM_DEPTH 4             // register sets of the load pipeline, up to 64 rows
#endif
#ifndef BATON_GEMM_DEPTH_WIDE
#define BATON_GEMM_DEPTH_WIDE 4        // past 64 rows
#endif

template <int MG, int KU, int NS>
void launch_skinny_mg(const baton::SkinnyArgs& a, dim3 grid, hipStream_t s) {
  constexpr int P = NS > 1 ? BATON_GEMM_DEPTH_WIDE : BATON_GEMM_DEPTH;
  const dim3 block(baton::kWave * baton::kGemmWaves);
  if (a.chunks == 1) hipLaunchKernelGGL((baton::skinny_gemm_kernel<MG, KU, 2, NS, P>), grid, block, 0, s, a);
  else hipLaunchKernelGGL((baton::skinny_gemm_kernel<MG, KU, 0, NS, P>), grid, block, 0, s, a);
}

// Row tiles, batch depth, slices per wave and row chunks for `rows` rows: up
// to 64 rows, one workgroup row set of ceil(rows / 16) tiles, one slice per
// wave and four 1 KB blocks per batch; past it, chunks of 64 rows with
// BATON_GEMM_NS_WIDE slices per wave (or, with BATON_GEMM_WIDE, all rows in
// one workgroup: 8 or 16 tiles with two or one block per batch).
int32_t row_chunks(int32_t rows) {
  return rows <= 64 || BATON_GEMM_WIDE ? 1 : (rows + 16 * BATON_GEMM_MG_WIDE - 1) / (16 * BATON_GEMM_MG_WIDE);
}
int32_t wave_slices(int32_t rows) { return rows <= 64 || BATON_GEMM_WIDE ? 1 : BATON_GEMM_NS_WIDE; }

// Workgroups of a grid of `groups` slice groups x `chunks` row chunks: with
// several chunks, whole sets of 8 groups (the kernel's XCD-aware dealing).
int64_t gemm_blocks(int32_t groups, int32_t chunks) {
  return chunks == 1 ? groups : (int64_t)(groups + 7) / 8 * 8 * chunks;
}

void launch_skinny(const baton::SkinnyArgs& a, dim3 grid, hipStream_t s) {
  const int32_t rows = a.rows;
  if (rows > 128 && BATON_GEMM_WIDE) return launch_skinny_mg<16, 1, 1>(a, grid, s);
  if (rows > 64 && BATON_GEMM_WIDE) return launch_skinny_mg<8, 2, 1>(a, grid, s);
  if (rows > 64) return launch_skinny_mg<BATON_GEMM_MG_WIDE, BATON_GEMM_KU_WIDE, BATON_GEMM_NS_WIDE>(a, grid, s);
  switch ((rows + 15) / 16) {
    case 1: return launch_skinny_mg<1, BATON_GEMM_KU, 1>(a, grid, s);
    case 2: return launch_skinny_mg<2, BATON_GEMM_KU, 1>(a, grid, s);
    case 3: return launch_skinny_mg<3, BATON_GEMM_KU, 1>(a, grid, s);
    default: return launch_skinny_mg<4, BATON_GEMM_KU, 1>(a, grid, s);
  }
}

}  // namespace

extern "C" {

size_t baton_linear_packed_bytes(int32_t out_dim, int32_t in_dim) {
  if (out_dim < 1 || in_dim < 1) return 0;
  return (size_t)((out_dim + 15) / 16) * 16 * (size_t)((in_dim + 31) / 32) * 32 * 2;
}

baton_status baton_linear_pack(int32_t dtype, const void* w, void* wp, int32_t out_dim, int32_t in_dim,
                               hipStream_t stream) {
  if (!w || !wp || out_dim < 1 || in_dim < 1 || in_dim % 8 || out_dim % 8) return BATON_EINVAL;
  if (dtype != BATON_BF16) return BATON_EDTYPE;
  if (!aligned16(w) || !aligned16(wp) || in_dim > (1 << 24)) return BATON_EINVAL;
  const int32_t kt = (in_dim + 31) / 32;
  const int64_t n_pieces = (int64_t)((out_dim + 15) / 16) * kt * baton::kWave;
  hipLaunchKernelGGL(baton::pack_weight_kernel, dim3((unsigned)((n_pieces + 255) / 256)), dim3(256), 0, stream,
                     static_cast<const baton::u32x4*>(w), static_cast<baton::u32x4*>(wp), out_dim, in_dim, kt,
                     n_pieces);
  return hipGetLastError() == hipSuccess ? BATON_OK : BATON_EHIP;
}

}  // extern "C"

namespace {

// baton_linear_packed, and with gain the RMS norm of its output rows into
// y_norm (the split sums added and each row normalised by one kernel when the
// product splits along k).
baton_status linear_packed(int32_t dtype, const void* x, const void* wp, void* y, int32_t rows, int32_t out_dim,
                           int32_t in_dim, int32_t accumulate, const void* gain, float eps, void* y_norm, void* ws,
                           size_t ws_bytes, hipStream_t stream) {
  if (!x || !wp || !y || rows < 1 || rows > BATON_GEMM_MAX_ROWS || out_dim < 1 || in_dim < 1 || (ws_bytes && !ws))
    return BATON_EINVAL;
  if (gain && (!y_norm || !aligned16(gain) || !aligned16(y_norm) || !(eps >= 0.f) || !std::isfinite(eps)))
    return BATON_EINVAL;
  if (accumulate != 0 && accumulate != 1) return BATON_EINVAL;
  if (dtype != BATON_BF16) return BATON_EDTYPE;
  if (!aligned16(x) || !aligned16(wp) || !aligned16(y) || in_dim % 8 || out_dim % 8 || in_dim > (1 << 24))
    return BATON_EINVAL;
  // 16-row weight slices, streamed by waves (one slice each up to 64 rows,
  // two past it) per 64-row chunk of x; with fewer than BATON_GEMM_MIN_SLICES
  // such waves (BATON_GEMM_MIN_WAVES_WIDE past 64 rows), split along k into
  // about BATON_GEMM_TARGET_WAVES(_WIDE) / waves ranges (at least 8 blocks of
  // 32 each, and only as many as the workspace holds partial sums for).
  // Measured on the llama2-7b shapes: at 64 rows the split's partial sums and
  // second launch cost more than they gain once the slices alone give two
  // waves per SIMD; past 64 rows the output and down projections (one or two
  // workgroups per CU unsplit) gain from it, the QKV projection at 128 rows
  // (768 waves) does not.
  const int32_t slices = (out_dim + 15) / 16, kt = (in_dim + 31) / 32, chunks = row_chunks(rows);
  const int32_t ns = wave_slices(rows), waves = (slices + ns - 1) / ns * chunks;
  const int32_t min_waves = chunks > 1 ? BATON_GEMM_MIN_WAVES_WIDE : BATON_GEMM_MIN_SLICES;
  const int32_t target = chunks > 1 ? BATON_GEMM_TARGET_WAVES_WIDE : BATON_GEMM_TARGET_WAVES;
  int32_t S = 1;
  if (waves < min_waves) S = std::max(1, std::min((target + waves - 1) / waves, kt / 8));
  if (!ws || !aligned16(ws)) S = 1;
  while (S > 1 && (size_t)S * rows * out_dim * sizeof(float) > ws_bytes) --S;
  const int32_t tc = (kt + S - 1) / S;
  S = (kt + tc - 1) / tc;
  baton::SkinnyArgs a;
  a.x = static_cast<const uint16_t*>(x);
  a.wp = static_cast<const uint16_t*>(wp);
  a.y = static_cast<uint16_t*>(y);
  a.part = static_cast<float*>(ws);
  a.rows = rows;
  a.N = out_dim;
  a.K = in_dim;
  a.kt = kt;
  a.tc = tc;
  a.accumulate = accumulate;
  a.gated = 0;
  a.chunks = chunks;
  a.groups = (slices + baton::kGemmWaves * ns - 1) / (baton::kGemmWaves * ns);
  const dim3 grid((unsigned)gemm_blocks(a.groups, chunks), (unsigned)S);
  launch_skinny(a, grid, stream);
  const int64_t n_out = (int64_t)rows * out_dim;
  if (S > 1 && gain) {
    hipLaunchKernelGGL(baton::reduce_rmsnorm_kernel, dim3(rows), dim3(baton::kRowThreads), 0, stream, a.part, a.y, S,
                       n_out, accumulate, static_cast<const baton::u32x4*>(gain),
                       static_cast<baton::u32x4*>(y_norm), out_dim / 8, 1.0f / out_dim, eps);
  } else {
    if (S > 1)
      hipLaunchKernelGGL(baton::gemm_reduce_kernel, dim3((unsigned)((n_out / 4 + 255) / 256)), dim3(256), 0, stream,
                         a.part, a.y, S, n_out, accumulate);
    if (gain)
      hipLaunchKernelGGL(baton::rmsnorm_kernel, dim3(rows), dim3(baton::kRowThreads), 0, stream,
                         static_cast<const baton::u32x4*>(y), static_cast<const baton::u32x4*>(gain),
                         static_cast<baton::u32x4*>(y_norm), out_dim / 8, 1.0f / out_dim, eps);
  }
  return hipGetLastError() == hipSuccess ? BATON_OK : BATON_EHIP;
}

}  // namespace

extern "C" {

baton_status baton_linear_packed(int32_t dtype, const void* x, const void* wp, void* y, int32_t rows,
                                 int32_t out_dim, int32_t in_dim, int32_t accumulate, void* ws, size_t ws_bytes,
                                 hipStream_t stream) {
  return linear_packed(dtype, x, wp, y, rows, out_dim, in_dim, accumulate, nullptr, 0.f, nullptr, ws, ws_bytes,
                       stream);
}

baton_status baton_linear_packed_rmsnorm(int32_t dtype, const void* x, const void* wp, void* y, int32_t rows,
                                         int32_t out_dim, int32_t in_dim, int32_t accumulate, const void* gain,
                                         float eps, void* y_norm, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!gain) return BATON_EINVAL;
  return linear_packed(dtype, x, wp, y, rows, out_dim, in_dim, accumulate, gain, eps, y_norm, ws, ws_bytes,
                       stream);
}

baton_status baton_linear_packed_silu(int32_t dtype, const void* x, const void* wp, void* y, int32_t rows,
                                      int32_t out_dim, int32_t in_dim, hipStream_t stream) {
  if (!x || !wp || !y || rows < 1 || rows > BATON_GEMM_MAX_ROWS || out_dim < 32 || out_dim % 32 || in_dim < 8 ||
      in_dim % 8 || in_dim > (1 << 24))
    return BATON_EINVAL;
  if (dtype != BATON_BF16) return BATON_EDTYPE;
  if (!aligned16(x) || !aligned16(wp) || !aligned16(y)) return BATON_EINVAL;
  baton::SkinnyArgs a;
  a.x = static_cast<const uint16_t*>(x);
  a.wp = static_cast<const uint16_t*>(wp);
  a.y = static_cast<uint16_t*>(y);
  a.part = nullptr;
  a.rows = rows;
  a.N = out_dim;
  a.K = in_dim;
  a.kt = (in_dim + 31) / 32;
  a.tc = a.kt;   // never split along k: the epilogue needs the whole sum
  a.accumulate = 0;
  a.gated = out_dim / 2;
  a.chunks = row_chunks(rows);
  const int32_t ns = wave_slices(rows);
  a.groups = (out_dim / 32 + 2 * ns - 1) / (2 * ns);   // 2 ns gate slices per workgroup
  const dim3 grid((unsigned)gemm_blocks(a.groups, a.chunks), 1);
  launch_skinny(a, grid, stream);
  return hipGetLastError() == hipSuccess ? BATON_OK : BATON_EHIP;
}

baton_status baton_rmsnorm(int32_t dtype, const void* x, const void* gain, void* y, int32_t rows, int32_t dim,
                           float eps, hipStream_t stream) {
  if (!x || !gain || !y || rows < 1 || dim < 8 || dim % 8 || !(eps >= 0.f) || !std::isfinite(eps)) return BATON_EINVAL;
  if (dtype != BATON_BF16) return BATON_EDTYPE;
  if (!aligned16(x) || !aligned16(gain) || !aligned16(y)) return BATON_EINVAL;
  hipLaunchKernelGGL(baton::rmsnorm_kernel, dim3(rows), dim3(baton::kRowThreads), 0, stream,
                     static_cast<const baton::u32x4*>(x), static_cast<const baton::u32x4*>(gain),
                     static_cast<baton::u32x4*>(y), dim / 8, 1.0f / dim, eps);
  return hipGetLastError() == hipSuccess ? BATON_OK : BATON_EHIP;
}

baton_status baton_silu_mul(int32_t dtype, const void* gate_up, void* out, int32_t rows, int32_t dim,
                            hipStream_t stream) {
  if (!gate_up || !out || rows < 1 || dim < 8 || dim % 8) return BATON_EINVAL;
  if (dtype != BATON_BF16) return BATON_EDTYPE;
  if (!aligned16(gate_up) || !aligned16(out)) return BATON_EINVAL;
  const int64_t n_vec = (int64_t)rows * (dim / 8);
  hipLaunchKernelGGL(baton::silu_mul_kernel, dim3((unsigned)((n_vec + 255) / 256)), dim3(256), 0, stream,
                     static_cast<const baton::u32x4*>(gate_up), static_cast<baton::u32x4*>(out), dim / 8, n_vec);
  return hipGetLastError() == hipSuccess ? BATON_OK : BATON_EHIP;
}

}  // extern "C"
