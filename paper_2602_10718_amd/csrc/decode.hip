// FP8 MLA decode kernel (Algorithm 1; Appendix D recurrences; Section 3.2).
//
// One workgroup = 4 waves = 64 query rows of one row group x a contiguous range
// of 64-token KV blocks (one page each).  Wave w owns row tile rt = w/2 (32 rows)
// and, for the PV product, the 256 latent dimensions dh = w%2.
//
// Data movement: every 64-token page (32 KiB E4M3 latent, 8 KiB bf16 RoPE,
// 256 B scales) is copied HBM -> LDS with 16-byte direct-to-LDS loads into a
// 3-stage ring, two pages ahead of the compute.  Latent rows are stored with the
// 16-byte chunk index XOR-swizzled by the token index so that both the
// token-major QK reads and the transposed PV reads avoid bank conflicts.
//
// Per block, per wave (all matrices transposed so that one lane owns one query
// row and the softmax statistics stay in registers):
//   S^T[64 tok x 32 rows]  = K_c^T . q8^T   (32x32x64 FP8 MFMA, K = 512)
//                          + K_r^T . q_r^T  (32x32x16 BF16 MFMA, K = 64)
//   s = log2(e) * tau * (sigma_q sigma_K acc_c + acc_r)   -- Section 3.1 alignment,
//       applied on the accumulators instead of pre-scaling the RoPE operands
//   online softmax, fused P' = e * sigma_K, block scale sigma_P, E4M3 codes
//   O^T[256 dims x 32 rows] = gamma * O^T + V^T . P'^T   (FP8 MFMA, K = 64 tokens)
// where V^T is read straight from the token-major latent tile with the LDS
// transpose read (ds_read_b64_tr_b8), the CDNA analogue of the paper's V-tile
// transposition, and the P codes are already in the B-operand layout (no
// permutation needed, the analogue of the paper's P-accumulator permutation).
// Blocks are visited in increasing order (the monotone order of Appendix E).

#include "snapmla_device.h"
#include "snapmla_internal.h"

namespace snapmla {

constexpr int kLatBytes = kPage * kDc;          // 32768
constexpr int kRopeBytes = kPage * kDr * 2;     // 8192
constexpr int kScBytes = kPage * 4;             // 256
constexpr int kStageBytes = kLatBytes + kRopeBytes + kScBytes;
constexpr int kStages = 3;
constexpr int kDmaPerBlock = 11;                // direct-to-LDS instructions per wave per page
constexpr float kLn2 = 0.69314718055994531f;

// Largest b with prefix[b] <= gb (prefix is non-decreasing, prefix[B] > gb).
__device__ __forceinline__ int find_seq(const int32_t* __restrict__ prefix, int B, int gb) {
  int lo = 0, hi = B - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (prefix[mid] <= gb) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Issue the copies of one page into an LDS stage.  Tokens at or past `valid`
// (slots after the end of the sequence) are read from the zero area instead, so
// the stage holds zero latent/RoPE/scale there.
__device__ __forceinline__ void issue_page(const DecodeArgs& a, int page, int valid, uint8_t* stage, int w,
                                           int lane) {
  const uint8_t* lat = a.kv_latent + (int64_t)page * kLatBytes;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int P = 64 * (8 * w + j) + lane;
    const int t = P >> 5, cp = P & 31;
    const uint8_t* src = t < valid ? lat + t * kDc + ((cp ^ (t & 31)) << 4) : a.zero + (cp << 4);
    g2lds16(src, stage + 1024 * (8 * w + j));
  }
  const uint8_t* rp = reinterpret_cast<const uint8_t*>(a.k_rope) + (int64_t)page * kRopeBytes;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int P = 64 * (2 * w + j) + lane;
    const int t = P >> 3, cp = P & 7;
    const uint8_t* src = t < valid ? rp + t * (kDr * 2) + ((cp ^ (t & 7)) << 4) : a.zero + (cp << 4);
    g2lds16(src, stage + kLatBytes + 1024 * (2 * w + j));
  }
  if (lane < 16) {
    const int t = 16 * w + lane;
    const float* src = t < valid ? a.kv_scale + (int64_t)page * kPage + t : reinterpret_cast<const float*>(a.zero);
    g2lds4(src, stage + kLatBytes + kRopeBytes + 64 * w);
  }
}

__global__ __launch_bounds__(256, 1) void decode_kernel(DecodeArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t smem[kStages * kStageBytes];

  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int rt = w >> 1, dh = w & 1;
  const int h = lane >> 5, n = lane & 31;

  const int g = blockIdx.x % a.G;
  const int unit = blockIdx.x / a.G;

  // ---- the global block range of this workgroup --------------------------
  int gstart, gend;
  if (a.chunk_blocks == 0) {
    const int64_t T = a.prefix[a.B];
    gstart = (int)((int64_t)unit * T / a.num_splits);
    gend = (int)((int64_t)(unit + 1) * T / a.num_splits);
  } else {
    const int b = unit / a.num_splits, s = unit % a.num_splits;
    const int nb = a.prefix[b + 1] - a.prefix[b];
    const int k0 = s * a.chunk_blocks;
    if (k0 >= nb) return;
    gstart = a.prefix[b] + k0;
    gend = a.prefix[b] + min(k0 + a.chunk_blocks, nb);
  }
  if (gstart >= gend) return;

  // loader cursor (sequence of the next block to copy)
  int ld_b = find_seq(a.prefix, a.B, gstart);
  int ld_gb = gstart;
  uint32_t stage_bad = 0;   // bit i: the page in stage i had an id out of range (wave-uniform)

  auto issue_next = [&](int stage_idx) {
    while (a.prefix[ld_b + 1] <= ld_gb) ++ld_b;
    const int blk = ld_gb - a.prefix[ld_b];
    int page = a.page_table[(int64_t)ld_b * a.max_pages + blk];
    const bool badp = page < 0 || page >= a.num_pages;
    if (badp) page = 0;
    stage_bad = (stage_bad & ~(1u << stage_idx)) | ((badp ? 1u : 0u) << stage_idx);
    const int valid = min(kPage, a.seq_lens[ld_b] - blk * kPage);
    issue_page(a, page, valid, smem + stage_idx * kStageBytes, w, lane);
    ++ld_gb;
  };

  const int nblocks = gend - gstart;
  issue_next(0);
  if (nblocks > 1) issue_next(1);

  // ---- per-piece state ---------------------------------------------------
  const int row = 64 * g + 32 * rt + n;       // row of this lane within the sequence
  const bool row_ok = row < a.R;
  const float LOG2E_TAU = a.sl2;

  int cur_b = -1, cur_nblk = 0, cur_blk0 = 0;
  bool cur_bad = false;
  int vis = 0;
  float cq = 0.f;                 // sigma_q * tau * log2(e)
  v8i qv[8];
  v4i qr[4];
  float m = -INFINITY, sp = 1.0f, l = 0.0f;
  v16f O[8];

  auto finish_piece = [&]() {
    const int piece = a.chunk_blocks == 0 ? unit + cur_b : cur_b * a.num_splits + (cur_blk0 / a.chunk_blocks);
    if (!row_ok) return;
    float* po = a.part_o + ((int64_t)piece * a.rows_pad + row) * kDc + 256 * dh + 4 * h;
    const bool empty = !(l > 0.0f);
    const float inv = empty ? 0.0f : 1.0f / l;
    const float nanv = __builtin_nanf("");
#pragma unroll
    for (int T = 0; T < 8; ++T) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v4f v;
        v[0] = O[T][4 * q + 0] * inv; v[1] = O[T][4 * q + 1] * inv;
        v[2] = O[T][4 * q + 2] * inv; v[3] = O[T][4 * q + 3] * inv;
        if (cur_bad) v = v4f{nanv, nanv, nanv, nanv};
        *reinterpret_cast<v4f*>(po + 32 * T + 8 * q) = v;
      }
    }
    if (dh == 0 && h == 0) {
      float lse = empty ? -INFINITY : (m + log2f(sp * l)) * kLn2;
      if (cur_bad) lse = nanv;
      a.part_lse[(int64_t)piece * a.rows_pad + row] = lse;
    }
  };

  // per-lane constant addressing for the transposed V reads
  const int q16 = lane & 15, tri = q16 >> 1, trb = q16 & 1, g16 = (lane >> 4) & 1;
  int tr_tok[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) tr_tok[c] = 16 * c + 8 * (tri >> 2) + 4 * h + (tri & 3);

  for (int k = 0; k < nblocks; ++k) {
    const int gb = gstart + k;
    // ---- sequence switch: finish the previous piece, load this sequence's queries
    if (cur_b < 0 || gb >= a.prefix[cur_b + 1]) {
      if (cur_b >= 0) finish_piece();
      int b = cur_b < 0 ? find_seq(a.prefix, a.B, gb) : cur_b + 1;
      while (a.prefix[b + 1] <= gb) ++b;
      cur_b = b;
      cur_blk0 = gb - a.prefix[b];
      cur_nblk = a.prefix[b + 1] - a.prefix[b];
      cur_bad = false;
      const int N = a.seq_lens[b];
      const int t = row / a.H;
      vis = a.causal ? N - a.q_len + 1 + t : N;
      if (row_ok) {
        const int64_t qrow = (int64_t)b * a.R + row;
        const v4i* src = reinterpret_cast<const v4i*>(a.q8 + qrow * kDc);
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          const v4i lo4 = src[4 * s + 2 * h], hi4 = src[4 * s + 2 * h + 1];
          qv[s] = v8i{lo4[0], lo4[1], lo4[2], lo4[3], hi4[0], hi4[1], hi4[2], hi4[3]};
        }
        const v4i* rsrc = reinterpret_cast<const v4i*>(a.q_rope + qrow * kDr);
#pragma unroll
        for (int s = 0; s < 4; ++s) qr[s] = rsrc[2 * s + h];
        cq = a.sq[qrow] * LOG2E_TAU;
      } else {
#pragma unroll
        for (int s = 0; s < 8; ++s) qv[s] = v8i{0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
        for (int s = 0; s < 4; ++s) qr[s] = v4i{0, 0, 0, 0};
        cq = 0.f;
      }
      m = -INFINITY; sp = 1.0f; l = 0.0f;
#pragma unroll
      for (int T = 0; T < 8; ++T) O[T] = v16f{0};
    }
    const int blk = gb - a.prefix[cur_b];

    // ---- wait for this block's page, release the oldest stage ------------
    if (k + 1 < nblocks) wait_vmcnt<kDmaPerBlock>(); else wait_vmcnt<0>();
    __syncthreads();
    if (k + 2 < nblocks) issue_next((k + 2) % kStages);
    cur_bad |= ((stage_bad >> (k % kStages)) & 1u) != 0;

    const uint8_t* st = smem + (k % kStages) * kStageBytes;
    const uint8_t* st_rope = st + kLatBytes;
    const float* st_sc = reinterpret_cast<const float*>(st + kLatBytes + kRopeBytes);

    // ---- S^T = K . Q^T for both 32-token tiles ---------------------------
    v16f accC[2], accR[2];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      accC[tt] = v16f{0};
      accR[tt] = v16f{0};
      const uint8_t* krow = st + (32 * tt + n) * kDc;
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const v4i lo4 = *reinterpret_cast<const v4i*>(krow + (((4 * s + 2 * h) ^ n) << 4));
        const v4i hi4 = *reinterpret_cast<const v4i*>(krow + (((4 * s + 2 * h + 1) ^ n) << 4));
        const v8i A = v8i{lo4[0], lo4[1], lo4[2], lo4[3], hi4[0], hi4[1], hi4[2], hi4[3]};
        accC[tt] = mfma_f8_32x32x64(A, qv[s], accC[tt]);
      }
      const uint8_t* rrow = st_rope + (32 * tt + n) * (kDr * 2);
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const v4i A = *reinterpret_cast<const v4i*>(rrow + (((2 * s + h) ^ (n & 7)) << 4));
        accR[tt] = mfma_bf16_32x32x16(A, qr[s], accR[tt]);
      }
    }

    // ---- restored logits, online softmax, scale fusion, P quantization ----
    // lane (row n, half h) holds tokens 32*tt + 8*(v/4) + 4*h + v%4, v = 0..15
    float sk[32];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const v4f f = *reinterpret_cast<const v4f*>(st_sc + 32 * tt + 8 * q + 4 * h);
        sk[16 * tt + 4 * q + 0] = f[0]; sk[16 * tt + 4 * q + 1] = f[1];
        sk[16 * tt + 4 * q + 2] = f[2]; sk[16 * tt + 4 * q + 3] = f[3];
      }
    float s2[32];
    const bool tail = (blk + 1) * kPage > vis;   // some token of this block is not visible to this row
    float mloc = -INFINITY;
#pragma unroll
    for (int p = 0; p < 32; ++p) {
      const int tt = p >> 4, v = p & 15;
      float x = accC[tt][v] * (cq * sk[p]) + accR[tt][v] * LOG2E_TAU;
      if (tail) {
        const int j = blk * kPage + 32 * tt + 8 * (v >> 2) + 4 * h + (v & 3);
        x = j < vis ? x : -INFINITY;
      }
      s2[p] = x;
      mloc = fmaxf(mloc, x);
    }
    const float mblk = xhalf_max(mloc);
    const float m_new = fmaxf(m, mblk);
    const bool live = m_new > -INFINITY;     // false: nothing visible yet for this row
    float lsum = 0.f, pmax = 0.f;
    float pp[32];
#pragma unroll
    for (int p = 0; p < 32; ++p) {
      const float e = live ? __builtin_amdgcn_exp2f(s2[p] - m_new) : 0.0f;
      lsum += e;
      pp[p] = e * sk[p];
      pmax = fmaxf(pmax, pp[p]);
    }
    lsum = xhalf_sum(lsum);
    pmax = xhalf_max(pmax);
    float gamma = 1.0f;
    v8i P8 = v8i{0, 0, 0, 0, 0, 0, 0, 0};
    if (mblk > -INFINITY) {
      const float sP = fmaxf(pmax / kFp8Max, kEps);
      const float inv = 1.0f / sP;
      gamma = __builtin_amdgcn_exp2f(m - m_new) * (sp / sP);
      l = gamma * l + lsum * inv;
      m = m_new;
      sp = sP;
#pragma unroll
      for (int d = 0; d < 8; ++d) {
        int wd = cvt_pk_e4m3(pp[4 * d + 0] * inv, pp[4 * d + 1] * inv, 0, false);
        wd = cvt_pk_e4m3(pp[4 * d + 2] * inv, pp[4 * d + 3] * inv, wd, true);
        P8[d] = wd;
      }
    }

    // ---- O^T = gamma * O^T + V^T . P^T over this wave's 256 dimensions -----
#pragma unroll
    for (int T = 0; T < 8; ++T) {
      const int chunk = 16 * dh + 2 * T + g16;
      v2i r[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int tok = tr_tok[c];
        r[c] = lds_read_tr8(st + tok * kDc + ((chunk ^ (tok & 31)) << 4) + 8 * trb);
      }
      const v8i A = v8i{r[0][0], r[0][1], r[1][0], r[1][1], r[2][0], r[2][1], r[3][0], r[3][1]};
      O[T] = O[T] * gamma;
      O[T] = mfma_f8_32x32x64(A, P8, O[T]);
    }
  }
  finish_piece();
  // drain: nothing outstanding (the last iteration waited for vmcnt 0)
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream) {
  const int units = a.chunk_blocks == 0 ? a.num_splits : a.B * a.num_splits;
  const int64_t grid = (int64_t)units * a.G;
  if (grid <= 0) return hipSuccess;
  if (grid > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL(decode_kernel, dim3((unsigned)grid), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace snapmla
