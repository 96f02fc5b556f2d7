// Fused fetch-and-dequantize of the paged FP8 cache into BF16 rows (Section 3.3,
// Fused-Fetch-Dequant: decode phases that reuse the cache at high precision --
// chunk prefill, prefix caching -- read the quantized cache and dequantize it in
// registers, in one pass, without a staging copy).
//
// Output row of token j of sequence b (row cu[b] + j, 576 bf16):
//   [0, 512)    bf16_rne( fp32( E4M3(code_i) * sigma_K ) )
//   [512, 576)  the cached RoPE key, bit for bit
// A token whose page id is outside [0, num_pages), and every token of a sequence
// longer than max_pages * 64, gets a row of 0x7FC0 (NaN).
//
// HBM-bound: 644 B read and 1,152 B written per token.  One 256-thread
// workgroup per (logical page, sequence); wave w owns tokens 16w..16w+15 of the
// page.  Per token a lane converts 8 codes (an 8-byte load) into 8 bf16 (one
// 16-byte store), so every load instruction reads one 512-byte latent row and
// every store writes one contiguous 1 KiB output span; the wave's 16 scales come
// in one scalar load.  All loads of a wave are issued before the first convert.

#include "snapmla_device.h"
#include "snapmla_internal.h"

namespace snapmla {

namespace {

constexpr int kRowElems = kDc + kDr;             // 576 bf16 per output row
constexpr uint32_t kNanPair = 0x7FC07FC0u;       // two canonical bf16 NaNs

// float32 -> bf16 bits, round to nearest, ties to even; NaN -> 0x7FC0
__device__ __forceinline__ uint32_t bf16_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) { return bf16_rne(lo) | (bf16_rne(hi) << 16); }

__global__ __launch_bounds__(256) void fetch_dequant_kernel(FetchArgs a) {
  const int b = blockIdx.y, pg = blockIdx.x;
  const int64_t r0 = a.cu[b];
  const int64_t n64 = (int64_t)a.cu[b + 1] - r0;
  if (n64 <= (int64_t)pg * kPage) return;                       // past the sequence (or n <= 0)
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int t0 = pg * kPage + 16 * w;                           // first token of this wave
  const int nt = (int)min<int64_t>(16, n64 - t0);               // tokens of this wave
  if (nt <= 0) return;
  const bool len_bad = n64 > (int64_t)a.max_pages * kPage;
  const int page = len_bad ? -1 : a.page_table[(int64_t)b * a.max_pages + pg];
  uint16_t* out = a.out + (r0 + t0) * kRowElems;
  if (page < 0 || page >= a.num_pages) {
    // NaN rows: this page's tokens; for a sequence longer than the page table
    // also those of pages pg + max_pages, pg + 2 max_pages, ... (the grid has
    // max_pages pages per sequence)
    const v4i nan4 = v4i{(int)kNanPair, (int)kNanPair, (int)kNanPair, (int)kNanPair};
    for (int64_t q = pg; q * kPage < n64; q += len_bad ? a.max_pages : n64) {
      const int64_t tq0 = q * kPage + 16 * w;
      const int ntq = (int)max<int64_t>(0, min<int64_t>(16, n64 - tq0));
      uint16_t* oq = a.out + (r0 + tq0) * kRowElems;
      for (int t = 0; t < ntq; ++t) {
        reinterpret_cast<v4i*>(oq + t * kRowElems)[lane] = nan4;
        if (lane < 8) reinterpret_cast<v4i*>(oq + t * kRowElems + kDc)[lane] = nan4;
      }
    }
    return;
  }
  const int64_t slot0 = (int64_t)page * kPage + 16 * w;         // cache slot of the wave's first token
  const uint8_t* lat = a.kv_latent + slot0 * kDc + 8 * lane;
  const float* sc = a.kv_scale + slot0;
  // latent codes: 8 bytes of each of the wave's tokens (rows past the end are not read)
  v2i c[16];
#pragma unroll
  for (int t = 0; t < 16; ++t) c[t] = t < nt ? *reinterpret_cast<const v2i*>(lat + t * kDc) : v2i{0, 0};
  // RoPE: 16 tokens x 128 B = 2 KiB, 16 bytes per lane in two rounds (token 8i + lane/8, chunk lane%8)
  const uint8_t* rp = reinterpret_cast<const uint8_t*>(a.k_rope) + slot0 * (kDr * 2);
  v4i r[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int t = 8 * i + (lane >> 3);
    r[i] = t < nt ? *reinterpret_cast<const v4i*>(rp + t * (kDr * 2) + 16 * (lane & 7)) : v4i{0, 0, 0, 0};
  }
  float s[16];
#pragma unroll
  for (int t = 0; t < 16; ++t) s[t] = sc[t];                   // uniform: one scalar load
#pragma unroll
  for (int t = 0; t < 16; ++t) {
    if (t < nt) {
      const v2f f0 = __builtin_amdgcn_cvt_pk_f32_fp8(c[t][0], false);
      const v2f f1 = __builtin_amdgcn_cvt_pk_f32_fp8(c[t][0], true);
      const v2f f2 = __builtin_amdgcn_cvt_pk_f32_fp8(c[t][1], false);
      const v2f f3 = __builtin_amdgcn_cvt_pk_f32_fp8(c[t][1], true);
      const float st = s[t];
      const v4i o = v4i{(int)pack_bf16(f0[0] * st, f0[1] * st), (int)pack_bf16(f1[0] * st, f1[1] * st),
                        (int)pack_bf16(f2[0] * st, f2[1] * st), (int)pack_bf16(f3[0] * st, f3[1] * st)};
      reinterpret_cast<v4i*>(out + t * kRowElems)[lane] = o;
    }
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int t = 8 * i + (lane >> 3);
    if (t < nt) reinterpret_cast<v4i*>(out + t * kRowElems + kDc)[lane & 7] = r[i];
  }
}

}  // namespace

hipError_t launch_fetch_dequant(const FetchArgs& a, hipStream_t stream) {
  if (a.B == 0) return hipSuccess;
  hipLaunchKernelGGL(fetch_dequant_kernel, dim3((unsigned)a.max_pages, (unsigned)a.B), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace snapmla
