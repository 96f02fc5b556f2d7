// Test hooks that expose single device operations the decode path relies on.

#include "snapmla.h"
#include "snapmla_device.h"
#include "snapmla_internal.h"

namespace snapmla {

// One 16x16x128 FP8 MFMA per tile (the instruction of the decode's QK content term):
// c[t][m][n] = sum_k A[t][m][k] B[t][n][k] over E4M3 codes, float32 accumulation
// from zero.  Lane (i % 16, i / 16) supplies K positions 32 (i / 16) .. +31 of row
// i % 16 of A and of B; C lane i register v is C[4 (i / 16) + v][i % 16].
__global__ __launch_bounds__(64) void mfma_fp8_kernel(const uint8_t* __restrict__ a, const uint8_t* __restrict__ b,
                                                      float* __restrict__ c, int64_t tiles) {
  const int64_t t = blockIdx.x;
  if (t >= tiles) return;
  const int lane = threadIdx.x, r = lane & 15, g = lane >> 4;
  const v4i* pa = reinterpret_cast<const v4i*>(a + t * 2048 + r * 128 + 32 * g);
  const v4i* pb = reinterpret_cast<const v4i*>(b + t * 2048 + r * 128 + 32 * g);
  const v4i a0 = pa[0], a1 = pa[1], b0 = pb[0], b1 = pb[1];
  v4f acc = v4f{0.f, 0.f, 0.f, 0.f};
  acc = mfma_f8_16x16x128(v8i{a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]},
                          v8i{b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]}, acc);
#pragma unroll
  for (int v = 0; v < 4; ++v) c[t * 256 + (4 * g + v) * 16 + r] = acc[v];
}

hipError_t launch_mfma_fp8(const uint8_t* a, const uint8_t* b, float* c, int64_t tiles, hipStream_t stream) {
  if (tiles <= 0) return hipSuccess;
  hipLaunchKernelGGL(mfma_fp8_kernel, dim3((unsigned)tiles), dim3(64), 0, stream, a, b, c, tiles);
  return hipGetLastError();
}

}  // namespace snapmla
