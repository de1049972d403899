/*
 * Host side of the workload generator: fills host arrays with the values of
 * wl_core.h.  Input generation only; shared by the oracle's inputs and by the
 * uploads of the GPU tests.
 */
#include <stddef.h>
#include <stdint.h>

#include "wl_core.h"

uint64_t wl_host_stream_key(uint64_t seed, uint64_t stream) { return wl_stream_key(seed, stream); }
uint64_t wl_host_draw(uint64_t key, uint64_t j) { return wl_draw(key, j); }
float wl_host_normal(uint64_t key, uint64_t c) { return wl_normal(key, c); }
uint16_t wl_host_bf16_rne(float f) { return wl_bf16_rne(f); }

/*
 * out[i0][i1][i2][i3] (contiguous) = value(c0 + i0*s0 + i1*s1 + i2*s2 + i3*s3),
 * stored as fp32 bits (code WL_F32) or bf16 bits (code WL_BF16).
 * Returns 0, or -1 on a bad code or shape.
 */
int wl_host_fill(uint64_t key, int code, void* out, int64_t n0, int64_t n1, int64_t n2,
                 int64_t n3, uint64_t c0, uint64_t s0, uint64_t s1, uint64_t s2, uint64_t s3) {
  if ((code != WL_F32 && code != WL_BF16) || n0 < 0 || n1 < 0 || n2 < 0 || n3 < 0) return -1;
  const int64_t rows = n0 * n1 * n2;
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    const int64_t i2 = r % n2, i1 = (r / n2) % n1, i0 = r / (n2 * n1);
    const uint64_t base = c0 + (uint64_t)i0 * s0 + (uint64_t)i1 * s1 + (uint64_t)i2 * s2;
    if (code == WL_F32) {
      float* o = (float*)out + r * n3;
      for (int64_t i3 = 0; i3 < n3; ++i3) o[i3] = wl_normal(key, base + (uint64_t)i3 * s3);
    } else {
      uint16_t* o = (uint16_t*)out + r * n3;
      for (int64_t i3 = 0; i3 < n3; ++i3) o[i3] = wl_bf16_rne(wl_normal(key, base + (uint64_t)i3 * s3));
    }
  }
  return 0;
}
