// Per-token FP8 quantization kernels: dense rows (query quantization), the fused
// quantize-on-append into paged slots, the split plan, and an E4M3 test hook.
//
// Per-token rule (Appendix C per-token quantization; Section 3.1 per-token
// granularity for the content latent only; Algorithm 1's amax/448 scale rule):
//   sigma = max(fp32(amax / 448), 2^-40),  code_i = E4M3_rne(fp32(x_i / sigma)).
// Both divisions are IEEE float32 divisions (hipcc's default division is
// correctly rounded), so codes and scales are reproducible bit for bit.

#include "snapmla_device.h"
#include "snapmla_internal.h"

namespace snapmla {

// One wave quantizes one 512-element bf16 row: lane l owns elements 8l..8l+7.
__device__ __forceinline__ void quantize_row_wave(const uint16_t* __restrict__ src, uint8_t* __restrict__ dst,
                                                  float* __restrict__ scale_out, int lane) {
  const uint4 raw = reinterpret_cast<const uint4*>(src)[lane];
  float x[8];
  x[0] = bf16_to_f32(raw.x & 0xFFFFu); x[1] = bf16_to_f32(raw.x >> 16);
  x[2] = bf16_to_f32(raw.y & 0xFFFFu); x[3] = bf16_to_f32(raw.y >> 16);
  x[4] = bf16_to_f32(raw.z & 0xFFFFu); x[5] = bf16_to_f32(raw.z >> 16);
  x[6] = bf16_to_f32(raw.w & 0xFFFFu); x[7] = bf16_to_f32(raw.w >> 16);
  float a = 0.0f;
#pragma unroll
  for (int i = 0; i < 8; ++i) a = fmaxf(a, fabsf(x[i]));
  a = wave_max(a);
  const float sigma = fmaxf(a / kFp8Max, kEps);
  float y[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) y[i] = clamp448(x[i] / sigma);
  int w0 = cvt_pk_e4m3(y[0], y[1], 0, false);
  w0 = cvt_pk_e4m3(y[2], y[3], w0, true);
  int w1 = cvt_pk_e4m3(y[4], y[5], 0, false);
  w1 = cvt_pk_e4m3(y[6], y[7], w1, true);
  reinterpret_cast<uint2*>(dst)[lane] = make_uint2((uint32_t)w0, (uint32_t)w1);
  if (lane == 0) *scale_out = sigma;
}

__global__ __launch_bounds__(256) void quantize_rows_kernel(const uint16_t* __restrict__ x, int64_t rows,
                                                            uint8_t* __restrict__ codes,
                                                            float* __restrict__ scale) {
  const int lane = threadIdx.x & 63;
  const int64_t nw = (int64_t)gridDim.x * 4;
  for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < rows; r += nw)
    quantize_row_wave(x + r * kDc, codes + r * kDc, scale + r, lane);
}

// Fused-K-Append (Section 3.3, Layer 1): quantize new token `tok` (token t of
// sequence b, tok = b*n_new + t) and write it, with its unscaled bf16 RoPE row
// and its scale, into its paged slot.  One wave per token.
__device__ __forceinline__ void append_token_wave(const uint16_t* __restrict__ c_kv_new,
                                                  const uint16_t* __restrict__ k_rope_new,
                                                  const int32_t* __restrict__ page_table,
                                                  const int32_t* __restrict__ seq_lens, int64_t tok, int n_new,
                                                  int max_pages, int num_pages, uint8_t* __restrict__ kv_latent,
                                                  float* __restrict__ kv_scale, uint16_t* __restrict__ k_rope,
                                                  int lane) {
  const int b = (int)(tok / n_new), t = (int)(tok % n_new);
  const int pos = seq_lens[b] - n_new + t;
  if (pos < 0 || pos >= max_pages * kPage) return;
  const int page = page_table[(int64_t)b * max_pages + pos / kPage];
  if (page < 0 || page >= num_pages) return;
  const int64_t slot = (int64_t)page * kPage + (pos % kPage);
  quantize_row_wave(c_kv_new + tok * kDc, kv_latent + slot * kDc, kv_scale + slot, lane);
  if (lane < 8)
    reinterpret_cast<uint4*>(k_rope + slot * kDr)[lane] = reinterpret_cast<const uint4*>(k_rope_new + tok * kDr)[lane];
}

__global__ __launch_bounds__(256) void append_kernel(const uint16_t* __restrict__ c_kv_new,
                                                     const uint16_t* __restrict__ k_rope_new,
                                                     const int32_t* __restrict__ page_table,
                                                     const int32_t* __restrict__ seq_lens, int B, int n_new,
                                                     int max_pages, int num_pages, uint8_t* __restrict__ kv_latent,
                                                     float* __restrict__ kv_scale, uint16_t* __restrict__ k_rope) {
  const int lane = threadIdx.x & 63;
  const int64_t tok = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (tok >= (int64_t)B * n_new) return;
  append_token_wave(c_kv_new, k_rope_new, page_table, seq_lens, tok, n_new, max_pages, num_pages, kv_latent,
                    kv_scale, k_rope, lane);
}

__global__ __launch_bounds__(256) void encode_kernel(const float* __restrict__ x, int64_t n,
                                                     uint8_t* __restrict__ codes) {
  const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (i + 3 < n) {
    const float4 v = *reinterpret_cast<const float4*>(x + i);
    int w = cvt_pk_e4m3(clamp448(v.x), clamp448(v.y), 0, false);
    w = cvt_pk_e4m3(clamp448(v.z), clamp448(v.w), w, true);
    *reinterpret_cast<uint32_t*>(codes + i) = (uint32_t)w;
  } else {
    for (int64_t k = i; k < n; ++k) codes[k] = (uint8_t)(cvt_pk_e4m3(clamp448(x[k]), 0.0f, 0, false) & 0xFF);
  }
}

// Query quantization (Fused-Q-Quant) over all rows, plus, in block 0, the split
// plan: prefix[b] = number of 64-token blocks of valid sequences before b, and the
// start descriptor of every split unit (kDesc* layout).
__global__ __launch_bounds__(256) void prep_kernel(PrepArgs a) {
  const int tid = threadIdx.x, lane = tid & 63;
  if (blockIdx.x == 0) {
    __shared__ int sums[256];
    __shared__ int lens[256];
    __shared__ int wsum[4];
    __shared__ int useq[kPlanTable + 1];
    const int per = (a.B + 255) / 256;
    const int b0 = tid * per, b1 = min(a.B, b0 + per);
    int local = 0;
    for (int b = b0; b < b1; ++b) {
      const int n = a.seq_lens[b];
      if (per == 1) lens[tid] = n;
      const bool ok = seq_len_ok(n, a.q_len, a.max_pages, a.chunk_blocks, a.num_splits);
      const int nb = (n + kPage - 1) / kPage;
      a.flags[b] = ok ? 0 : 1;
      local += ok ? nb : 0;
    }
    // inclusive scan of the per-thread block counts: within each wave, then the four
    // wave totals
    int incl = local;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int v = __shfl_up(incl, off, 64);
      if (lane >= off) incl += v;
    }
    if (lane == 63) wsum[tid >> 6] = incl;
    __syncthreads();
    for (int i = 0; i < (tid >> 6); ++i) incl += wsum[i];
    sums[tid] = incl;
    if (tid == 0) a.prefix[0] = 0;
    if (per == 1) {
      if (tid < a.B) a.prefix[tid + 1] = incl;      // one sequence per thread: the scan is the prefix
    } else {
      int run = incl - local;
      for (int b = b0; b < b1; ++b) {
        const int n = a.seq_lens[b];
        run += a.flags[b] ? 0 : (n + kPage - 1) / kPage;
        a.prefix[b + 1] = run;
      }
    }
    reinterpret_cast<uint32_t*>(a.zero)[tid] = 0u;   // 256 threads x 4 B = 1 KiB
    if (tid == 0) a.ctrl[0] = a.out != nullptr ? 1 : 0;
    __syncthreads();                                 // prefix complete (LDS and global)

    // ---- start descriptors, one unit per thread ----------------------------
    // (with one sequence per thread, B <= 256, the scan's LDS sums are the prefix)
    const int T = sums[255];
    auto pref = [&](int i) { return per == 1 ? (i == 0 ? 0 : sums[i - 1]) : a.prefix[i]; };
    auto seq_of_block = [&](int gb) {                // largest b with prefix[b] <= gb
      int lo = 0, hi = a.B - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (pref(mid) <= gb) lo = mid; else hi = mid - 1;
      }
      return lo;
    };
    // balanced plan over virtual positions (kPlanPad): sequence b spans [V_b, V_b+1),
    // V_b = prefix[b] + pad*b, its real blocks after its first pad positions
    const int W = a.num_splits;
    const int64_t TV = (int64_t)T + (int64_t)a.pad * a.B;
    auto vstart = [&](int b) { return (int64_t)pref(b) + (int64_t)a.pad * b; };
    auto real_in = [&](int b, int64_t v) {           // real blocks before v, v in b's span
      const int p0 = pref(b);
      const int64_t r = v - vstart(b) - a.pad;
      return p0 + (int)(r < 0 ? 0 : min<int64_t>(r, pref(b + 1) - p0));
    };
    // with few enough units, every sequence (one per thread) marks the units whose
    // virtual start falls in its span: u with ceil(V_b W / TV) <= u < ceil(V_b+1 W / TV)
    const bool table = a.chunk_blocks == 0 && per == 1 && a.units <= kPlanTable && TV > 0;
    if (table) {
      if (tid < a.B) {
        const int ulo = (int)((vstart(tid) * W + TV - 1) / TV);
        const int uhi = (int)((vstart(tid + 1) * W + TV - 1) / TV);
        for (int u = ulo; u < uhi; ++u) useq[u] = tid;
      }
      __syncthreads();
    }
    for (int u = tid; u < a.units; u += 256) {
      int32_t* d = a.desc + (int64_t)u * kDescInts;
      int gs = 0, ge = 0, b = 0;
      if (a.chunk_blocks == 0) {
        if (TV > 0) {
          const int64_t vs = (int64_t)u * TV / W, ve = (int64_t)(u + 1) * TV / W;
          int bs, be;
          if (table) {
            bs = useq[u];
            be = u + 1 < W ? useq[u + 1] : a.B - 1;
          } else {                                   // largest b with V_b <= v
            auto seq_of_v = [&](int64_t v) {
              int lo = 0, hi = a.B - 1;
              while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (vstart(mid) <= v) lo = mid; else hi = mid - 1;
              }
              return lo;
            };
            bs = seq_of_v(vs);
            be = seq_of_v(ve);
          }
          gs = real_in(bs, vs);
          ge = real_in(be, ve);
          // block gs lies in sequence bs unless bs has no blocks
          if (gs < ge) b = pref(bs + 1) > gs ? bs : seq_of_block(gs);
        }
      } else {
        b = u / a.num_splits;
        const int64_t k0 = (int64_t)(u % a.num_splits) * a.chunk_blocks;
        const int p0 = pref(b), nb = pref(b + 1) - p0;
        if (k0 < nb) {
          gs = p0 + (int)k0;
          ge = p0 + (int)min<int64_t>(k0 + a.chunk_blocks, nb);
        }
      }
      d[kDescStart] = gs;
      d[kDescEnd] = ge;
      if (gs >= ge) continue;
      const int p0 = pref(b), p1 = pref(b + 1);
      d[kDescSeq] = b;
      d[kDescP0] = p0;
      d[kDescP1] = p1;
      d[kDescLen] = per == 1 ? lens[b] : a.seq_lens[b];
    }
    return;
  }
  if ((int)blockIdx.x <= a.ablocks) {              // fused quantize-on-append
    const int64_t tok = (int64_t)(blockIdx.x - 1) * 4 + (tid >> 6);
    if (tok < (int64_t)a.B * a.n_new)
      append_token_wave(a.c_kv_new, a.k_rope_new, a.page_table, a.seq_lens, tok, a.n_new, a.max_pages, a.num_pages,
                        a.kv_latent, a.kv_scale, a.k_rope, lane);
    return;
  }
  const int q0 = 1 + a.ablocks;                    // first row workgroup
  const int64_t nw = (int64_t)(gridDim.x - q0) * 4;
  for (int64_t r = (int64_t)(blockIdx.x - q0) * 4 + (tid >> 6); r < a.rows; r += nw) {
    // (the length is loaded first so that its round trip overlaps the quantization's)
    const int n = a.out != nullptr ? a.seq_lens[r / a.R] : 0;
    if (a.quantize) quantize_row_wave(a.q_nope + r * kDc, a.q8 + r * kDc, a.sq + r, lane);
    if (a.out != nullptr) {
      // a row of a sequence without blocks is final here: 0 and -inf for an empty
      // sequence, NaN for one a data error rejects (the decode writes no piece for it)
      const bool ok = seq_len_ok(n, a.q_len, a.max_pages, a.chunk_blocks, a.num_splits);
      if (!ok || n == 0) {
        const float v = ok ? 0.0f : __builtin_nanf("");
        if (a.out_dtype == 1) {
          v4f* dst = reinterpret_cast<v4f*>(static_cast<float*>(a.out) + r * kDc) + 2 * lane;
          dst[0] = v4f{v, v, v, v};
          dst[1] = v4f{v, v, v, v};
        } else {
          const int bv = ok ? 0 : 0x7FC0;
          reinterpret_cast<v4i*>(static_cast<uint16_t*>(a.out) + r * kDc)[lane] =
              v4i{bv | (bv << 16), bv | (bv << 16), bv | (bv << 16), bv | (bv << 16)};
        }
        if (a.out_lse != nullptr && lane == 0) a.out_lse[r] = ok ? -INFINITY : __builtin_nanf("");
      }
    }
  }
}

static int grid_for(int64_t waves) {
  int64_t g = (waves + 3) / 4;
  return (int)(g < 1 ? 1 : (g > 65535 ? 65535 : g));
}

hipError_t launch_quantize_rows(const uint16_t* x, int64_t rows, uint8_t* codes, float* scale,
                                hipStream_t stream) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(quantize_rows_kernel, dim3(grid_for(rows)), dim3(256), 0, stream, x, rows, codes, scale);
  return hipGetLastError();
}

hipError_t launch_append(const uint16_t* c_kv_new, const uint16_t* k_rope_new, const int32_t* page_table,
                         const int32_t* seq_lens, int B, int n_new, int max_pages, int num_pages,
                         uint8_t* kv_latent, float* kv_scale, uint16_t* k_rope, hipStream_t stream) {
  const int64_t toks = (int64_t)B * n_new;
  if (toks <= 0) return hipSuccess;
  const int64_t blocks = (toks + 3) / 4;
  if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL(append_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, c_kv_new, k_rope_new, page_table,
                     seq_lens, B, n_new, max_pages, num_pages, kv_latent, kv_scale, k_rope);
  return hipGetLastError();
}

hipError_t launch_encode(const float* x, int64_t n, uint8_t* codes, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 1023) / 1024;
  if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL(encode_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, x, n, codes);
  return hipGetLastError();
}

hipError_t launch_prep(const PrepArgs& a, hipStream_t stream) {
  const int qblocks = a.rows > 0 ? grid_for(a.rows) : 0;
  if ((int64_t)1 + a.ablocks + qblocks > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL(prep_kernel, dim3(1 + a.ablocks + qblocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace snapmla
