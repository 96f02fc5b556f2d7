// KV-cache quantizers of the accuracy ablation (Appendix G, Table 3): the batch's
// bf16 cache rows written into the paged planes under one of five granularities,
// so that the decode path can run on each and its error against BF16 attention
// can be compared.  Scale rule everywhere: sigma = max(fp32(amax / 448), 2^-40)
// over the configuration's group; codes = E4M3(fp32(x / sigma)), IEEE divisions.
//   0  per-token content, RoPE copied            (the method, as snapmla_quantize_append)
//   1  per-token over content and RoPE together, RoPE quantized with that scale and
//      stored back as bf16(fp32(sigma * E4M3(r / sigma)))          (RoPE-unaware)
//   2  per-tensor static: sigma = 1
//   3  per-tensor dynamic: one sigma from the amax of every content value of the batch
//   4  per-block: one sigma per 64-token page of a sequence
// Launch shape: one 256-thread workgroup per (logical page, sequence), a wave per 16
// tokens; tokens past a sequence's end, past the page table or with a page id outside
// [0, num_pages) are skipped.  Configuration 3 first reduces the batch amax into a
// caller-provided word (vector atomics on the float bits: amax >= 0 orders like an
// unsigned integer), configuration 4 first writes each page's scale into kv_scale.

#include "snapmla_device.h"
#include "snapmla_internal.h"

namespace snapmla {

namespace {

struct AblArgs {
  const uint16_t* c_kv;      // [T][512] bf16, token j of sequence b at row cu[b] + j
  const uint16_t* k_rope;    // [T][64]
  const int32_t* page_table;
  const int32_t* cu;
  uint32_t* amax_word;       // config 3
  uint8_t* kv_latent;
  float* kv_scale;
  uint16_t* k_rope_out;
  int B, max_pages, num_pages, config;
};

// The page of sequence b covered by this workgroup, or -1 when there is nothing to do.
__device__ __forceinline__ int block_page(const AblArgs& a, int b, int pg, int64_t& r0, int& n) {
  r0 = a.cu[b];
  const int64_t n64 = (int64_t)a.cu[b + 1] - r0;
  n = (int)min<int64_t>(n64, (int64_t)a.max_pages * kPage);
  if (n <= pg * kPage) return -1;
  const int page = a.page_table[(int64_t)b * a.max_pages + pg];
  return (page < 0 || page >= a.num_pages) ? -1 : page;
}

__device__ __forceinline__ float row_amax8(const uint16_t* row, int lane, float* x) {
  const uint4 raw = reinterpret_cast<const uint4*>(row)[lane];
  x[0] = bf16_to_f32(raw.x & 0xFFFFu); x[1] = bf16_to_f32(raw.x >> 16);
  x[2] = bf16_to_f32(raw.y & 0xFFFFu); x[3] = bf16_to_f32(raw.y >> 16);
  x[4] = bf16_to_f32(raw.z & 0xFFFFu); x[5] = bf16_to_f32(raw.z >> 16);
  x[6] = bf16_to_f32(raw.w & 0xFFFFu); x[7] = bf16_to_f32(raw.w >> 16);
  float m = 0.0f;
#pragma unroll
  for (int i = 0; i < 8; ++i) m = fmaxf(m, fabsf(x[i]));
  return m;
}

__global__ void abl_clear_kernel(uint32_t* w) { *w = 0u; }

// config 3: the amax of every content value of the batch (one atomic per workgroup)
__global__ __launch_bounds__(256) void abl_tensor_amax_kernel(AblArgs a) {
  __shared__ float wmax[4];
  int64_t r0;
  int n;
  const int page = block_page(a, blockIdx.y, blockIdx.x, r0, n);
  if (page < 0) return;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  float m = 0.0f, x[8];
  for (int t = 16 * w; t < 16 * w + 16; ++t) {
    const int j = blockIdx.x * kPage + t;
    if (j < n) m = fmaxf(m, row_amax8(a.c_kv + (r0 + j) * kDc, lane, x));
  }
  m = wave_max(m);
  if (lane == 0) wmax[w] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    const float blk = fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]));
    __hip_atomic_fetch_max(a.amax_word, __float_as_uint(blk), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// config 4: the scale of each 64-token page, written to its 64 slots of kv_scale
__global__ __launch_bounds__(256) void abl_block_scale_kernel(AblArgs a) {
  __shared__ float wmax[4];
  int64_t r0;
  int n;
  const int page = block_page(a, blockIdx.y, blockIdx.x, r0, n);
  if (page < 0) return;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  float m = 0.0f, x[8];
  for (int t = 16 * w; t < 16 * w + 16; ++t) {
    const int j = blockIdx.x * kPage + t;
    if (j < n) m = fmaxf(m, row_amax8(a.c_kv + (r0 + j) * kDc, lane, x));
  }
  m = wave_max(m);
  if (lane == 0) wmax[w] = m;
  __syncthreads();
  const float blk = fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]));
  if (threadIdx.x < kPage) a.kv_scale[(int64_t)page * kPage + threadIdx.x] = fmaxf(blk / kFp8Max, kEps);
}

__global__ __launch_bounds__(256) void abl_quant_kernel(AblArgs a) {
  int64_t r0;
  int n;
  const int page = block_page(a, blockIdx.y, blockIdx.x, r0, n);
  if (page < 0) return;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int t = 16 * w; t < 16 * w + 16; ++t) {
    const int j = blockIdx.x * kPage + t;
    if (j >= n) break;
    const int64_t row = r0 + j, slot = (int64_t)page * kPage + t;
    float x[8];
    const float cm = wave_max(row_amax8(a.c_kv + row * kDc, lane, x));
    // RoPE element of this lane (lanes 0..31 hold 2 each)
    float r0f = 0.0f, r1f = 0.0f;
    if (lane < 32) {
      const uint32_t rr = reinterpret_cast<const uint32_t*>(a.k_rope + row * kDr)[lane];
      r0f = bf16_to_f32(rr & 0xFFFFu);
      r1f = bf16_to_f32(rr >> 16);
    }
    float sigma;
    if (a.config == 0) {
      sigma = fmaxf(cm / kFp8Max, kEps);
    } else if (a.config == 1) {
      const float rm = wave_max(fmaxf(fabsf(r0f), fabsf(r1f)));
      sigma = fmaxf(fmaxf(cm, rm) / kFp8Max, kEps);
    } else if (a.config == 2) {
      sigma = 1.0f;
    } else if (a.config == 3) {
      const float am = __uint_as_float(__hip_atomic_load(a.amax_word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
      sigma = fmaxf(am / kFp8Max, kEps);
    } else {
      sigma = a.kv_scale[slot];
    }
    float y[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) y[i] = clamp448(x[i] / sigma);
    int w0 = cvt_pk_e4m3(y[0], y[1], 0, false);
    w0 = cvt_pk_e4m3(y[2], y[3], w0, true);
    int w1 = cvt_pk_e4m3(y[4], y[5], 0, false);
    w1 = cvt_pk_e4m3(y[6], y[7], w1, true);
    reinterpret_cast<uint2*>(a.kv_latent + slot * kDc)[lane] = make_uint2((uint32_t)w0, (uint32_t)w1);
    if (lane == 0) a.kv_scale[slot] = sigma;
    if (lane < 32) {
      uint32_t outw;
      if (a.config == 1) {
        const int c = cvt_pk_e4m3(clamp448(r0f / sigma), clamp448(r1f / sigma), 0, false);
        const v2f d = __builtin_amdgcn_cvt_pk_f32_fp8(c, false);
        const float q0 = d[0] * sigma, q1 = d[1] * sigma;
        auto rne = [](float v) -> uint32_t {
          const uint32_t u = __float_as_uint(v);
          if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
          return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
        };
        outw = rne(q0) | (rne(q1) << 16);
      } else {
        outw = reinterpret_cast<const uint32_t*>(a.k_rope + row * kDr)[lane];
      }
      reinterpret_cast<uint32_t*>(a.k_rope_out + slot * kDr)[lane] = outw;
    }
  }
}

}  // namespace

hipError_t launch_quantize_cache_config(const uint16_t* c_kv, const uint16_t* k_rope, const int32_t* page_table,
                                        const int32_t* cu, int B, int max_pages, int num_pages, int config,
                                        uint32_t* amax_word, uint8_t* kv_latent, float* kv_scale,
                                        uint16_t* k_rope_out, hipStream_t stream) {
  if (B == 0) return hipSuccess;
  AblArgs a{c_kv, k_rope, page_table, cu, amax_word, kv_latent, kv_scale, k_rope_out, B, max_pages, num_pages, config};
  const dim3 grid((unsigned)max_pages, (unsigned)B);
  if (config == 3) {
    hipLaunchKernelGGL(abl_clear_kernel, dim3(1), dim3(1), 0, stream, amax_word);
    hipLaunchKernelGGL(abl_tensor_amax_kernel, grid, dim3(256), 0, stream, a);
  } else if (config == 4) {
    hipLaunchKernelGGL(abl_block_scale_kernel, grid, dim3(256), 0, stream, a);
  }
  hipLaunchKernelGGL(abl_quant_kernel, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace snapmla
