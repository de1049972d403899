// Device side of the workload generator: the same values as wl_host.c, written
// straight into HBM so that multi-GB inputs never cross PCIe.  Input
// generation only; no step of the re-batching method lives here.
#include <hip/hip_runtime.h>
#include <stdint.h>

#define WL_QUAL __device__ static inline
#include "wl_core.h"

namespace {

// Threads stride over the innermost two dimensions; (blockIdx.y, blockIdx.z)
// name one row of the flattened outer two dimensions.
template <int CODE>
__global__ void __launch_bounds__(256) wl_fill_kernel(uint64_t key, void* __restrict__ out,
                                                      int64_t n_outer, int64_t n1, int64_t n2,
                                                      int64_t n3, uint64_t c0, uint64_t s0,
                                                      uint64_t s1, uint64_t s2, uint64_t s3) {
  const int64_t inner = n2 * n3;
  const int64_t outer = (int64_t)blockIdx.y + (int64_t)gridDim.y * blockIdx.z;
  if (outer >= n_outer) return;
  const int64_t i0 = outer / n1, i1 = outer % n1;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < inner;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i2 = e / n3, i3 = e % n3;
    const uint64_t c = c0 + (uint64_t)i0 * s0 + (uint64_t)i1 * s1 + (uint64_t)i2 * s2 +
                       (uint64_t)i3 * s3;
    const float x = wl_normal(key, c);
    const int64_t o = outer * inner + e;
    if (CODE == WL_F32) {
      reinterpret_cast<float*>(out)[o] = x;
    } else {
      reinterpret_cast<uint16_t*>(out)[o] = wl_bf16_rne(x);
    }
  }
}

// Read-only HBM stream: each workgroup reads one 64 KiB chunk with 16-byte
// non-temporal loads, eight in flight per thread, and folds them so the loads
// are kept; the flag is written only if the fold hits a fixed value.  A
// measurement reference for the bandwidth plain reads reach, not a step of
// the method.
typedef uint32_t wl_u32x4 __attribute__((ext_vector_type(4)));

__global__ void __launch_bounds__(256) wl_read_kernel(const wl_u32x4* __restrict__ buf, uint32_t* flag) {
  const wl_u32x4* chunk = buf + (int64_t)blockIdx.x * 4096;
  uint32_t x = 0;
  for (int i = threadIdx.x; i < 4096; i += 256 * 8) {
    wl_u32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(chunk + i + 256 * u);
#pragma unroll
    for (int u = 0; u < 8; ++u) x ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  if (x == 0x9E3779B9u) flag[0] = x;
}

}  // namespace

extern "C" {

// Enqueues one read of `bytes` (a multiple of 64 KiB) of device memory buf
// (16-byte aligned); flag: one device uint32 the kernel may write.  Returns
// 0, -1 on bad arguments, or the hipError_t.
int wl_device_read_stream(const void* buf, int64_t bytes, uint32_t* flag, hipStream_t stream) {
  if (!buf || !flag || bytes <= 0 || bytes % 65536 || (reinterpret_cast<uintptr_t>(buf) & 15) ||
      bytes / 65536 > 0x7FFFFFFF)
    return -1;
  hipLaunchKernelGGL(wl_read_kernel, dim3((unsigned)(bytes / 65536)), dim3(256), 0, stream,
                     static_cast<const wl_u32x4*>(buf), flag);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

// Device twin of wl_host_fill: out is device memory laid out [n0][n1][n2][n3].
// Enqueued on `stream`; returns 0, -1 on bad arguments, or the hipError_t.
int wl_device_fill(uint64_t key, int code, void* out, int64_t n0, int64_t n1, int64_t n2,
                   int64_t n3, uint64_t c0, uint64_t s0, uint64_t s1, uint64_t s2,
                   uint64_t s3, hipStream_t stream) {
  if ((code != WL_F32 && code != WL_BF16) || n0 < 0 || n1 < 0 || n2 < 0 || n3 < 0) return -1;
  const int64_t outer = n0 * n1, inner = n2 * n3;
  if (outer == 0 || inner == 0) return 0;
  if (out == nullptr) return -1;
  // Outer rows are spread over (y, z) to stay under the 65535 grid limit;
  // blocks past the last row return at once.
  const int64_t by = outer < 65535 ? outer : 65535;
  const int64_t bz = (outer + by - 1) / by;
  if (bz > 65535) return -1;
  int64_t bx = (inner + 255) / 256;
  if (bx > 2048) bx = 2048;
  dim3 grid((unsigned)bx, (unsigned)by, (unsigned)bz);
  if (code == WL_F32)
    hipLaunchKernelGGL(wl_fill_kernel<WL_F32>, grid, dim3(256), 0, stream, key, out, outer, n1,
                       n2, n3, c0, s0, s1, s2, s3);
  else
    hipLaunchKernelGGL(wl_fill_kernel<WL_BF16>, grid, dim3(256), 0, stream, key, out, outer, n1,
                       n2, n3, c0, s0, s1, s2, s3);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

}  // extern "C"
