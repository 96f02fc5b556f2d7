// FP8 MLA decode kernel (Algorithm 1; Appendix D recurrences; Section 3.2).
//
// One workgroup = 8 waves (two per SIMD) = 64 query rows of one row group x a
// contiguous range of 64-token KV blocks (one page each).  The waves specialise:
//   QK waves  w = 0..3, (rt, tt) = (w/2, w%2): S^T tile of row tile rt (32 rows)
//             and token tile tt (tokens 32tt..32tt+31), online softmax, scale
//             fusion and E4M3 probability codes; they own q and the row state.
//   PV waves  w = 4..7, (rt, dh) = ((w-4)/2, (w-4)%2): O^T of row tile rt and
//             latent dimensions 256dh..256dh+255; they own the output accumulator.
// The two QK waves of a row tile exchange tile statistics through LDS and
// publish the probability codes and the per-row rescale factor; the PV waves
// consume them one block later.  So on every SIMD a QK wave works on block k
// while a PV wave works on block k-1, with two workgroup barriers per block.
// (The paper's Hopper kernel splits the work between two warp groups, Algorithm 1
// and Appendix E; here the split is by phase instead of by output half.)
//
// Data movement: each 64-token page (32 KiB E4M3 latent, 8 KiB bf16 RoPE,
// 256 B scales) is copied HBM -> LDS with 16-byte direct-to-LDS loads into a
// 3-stage ring, two pages ahead of the compute.  Latent rows are stored with the
// 16-byte chunk index XOR-swizzled by the token index so that both the
// token-major QK reads and the transposed PV reads avoid bank conflicts.
//
// Per block (matrices transposed so that one lane owns one query row):
//   S^T[32 tok x 32 rows]  = K_c^T . q8^T   (32x32x64 FP8 MFMA, K = 512)
//                          + K_r^T . q_r^T  (32x32x16 BF16 MFMA, K = 64)
//   s = log2(e) tau (sigma_q sigma_K acc_c + acc_r)   (Section 3.1 domain alignment,
//       applied to the two accumulators instead of pre-scaling the RoPE operands)
//   running max m, block scale sigma_P = max(max(e sigma_K) / 448, 2^-40),
//   gamma = exp(m_old - m) sigma_p_old / sigma_P, l = gamma l + sum(e) / sigma_P,
//   codes pi = E4M3(e sigma_K / sigma_P)                 (Appendix D)
//   O^T[256 dims x 32 rows] = gamma O^T + V^T . P^T       (FP8 MFMA, K = 64 tokens)
// V^T is read straight from the token-major latent tile with the LDS transpose
// read (ds_read_b64_tr_b8; the CDNA counterpart of the paper's V-tile
// transposition) and the P codes are already in the B-operand layout, so no
// accumulator permutation is needed.  Blocks are consumed in increasing order,
// the monotone order of Appendix E.

#include "snapmla_device.h"
#include "snapmla_internal.h"

namespace snapmla {

constexpr int kLatBytes = kPage * kDc;          // 32768
constexpr int kRopeBytes = kPage * kDr * 2;     // 8192
constexpr int kScBytes = kPage * 4;             // 256
constexpr int kStageBytes = kLatBytes + kRopeBytes + kScBytes;
constexpr int kStages = 3;
constexpr int kWaves = 8;
constexpr int kDmaPerBlock = 6;                 // direct-to-LDS instructions per wave per page
constexpr int kXsBytes = 2 * 2 * 32 * 16;       // tile statistics [rt][tt][row] x float4
constexpr int kXcBytes = 2 * 2 * 64 * 16;       // probability codes [rt][tt][lane] x 16 B
constexpr int kXgBytes = 2 * 32 * 16;           // per-row gamma and l [rt][row] x float4
constexpr int kSmemBytes = kStages * kStageBytes + kXsBytes + kXcBytes + kXgBytes;
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

__device__ __forceinline__ const void* sel_ptr(bool c, const void* a, const void* b) {
  const uint64_t m = 0ull - (uint64_t)c;
  return reinterpret_cast<const void*>((reinterpret_cast<uint64_t>(a) & m) | (reinterpret_cast<uint64_t>(b) & ~m));
}

// This wave's share of the copies of one page into an LDS stage.  Tokens at or
// past `valid` (slots after the end of the sequence) are read from the zero area
// instead, so the stage holds zero latent/RoPE/scale there.
__device__ __forceinline__ void issue_page(const uint8_t* __restrict__ lat_base, const uint8_t* __restrict__ rope_base,
                                           const float* __restrict__ sc_base, const uint8_t* zero, int page, int valid,
                                           uint8_t* stage, int w, int lane) {
  const uint8_t* lat = lat_base + (int64_t)page * kLatBytes;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int P = 64 * (4 * w + j) + lane;
    const int t = P >> 5, cp = P & 31;
    g2lds16(sel_ptr(t < valid, lat + t * kDc + ((cp ^ (t & 31)) << 4), zero + (cp << 4)),
            stage + 1024 * (4 * w + j));
  }
  {
    const int P = 64 * w + lane;
    const int t = P >> 3, cp = P & 7;
    g2lds16(sel_ptr(t < valid, rope_base + (int64_t)page * kRopeBytes + t * (kDr * 2) + ((cp ^ (t & 7)) << 4),
                    zero + (cp << 4)),
            stage + kLatBytes + 1024 * w);
  }
  if (lane < 8) {
    const int t = 8 * w + lane;
    g2lds4(sel_ptr(t < valid, sc_base + (int64_t)page * kPage + t, zero), stage + kLatBytes + kRopeBytes + 32 * w);
  }
}

// Top-of-block barrier: the page of this block has landed (the next page may still
// be in flight unless `drain`), and every LDS write of the previous phase is visible.
__device__ __forceinline__ void block_barrier(bool drain) {
  if (drain) barrier_vm_lgkm0<0>(); else barrier_vm_lgkm0<kDmaPerBlock>();
}

__global__ __launch_bounds__(512, 1) void decode_kernel(DecodeArgs a, const int32_t* __restrict__ prefix,
                                                        const int32_t* __restrict__ page_table,
                                                        const int32_t* __restrict__ seq_lens) {
  __shared__ __attribute__((aligned(1024))) uint8_t smem[kSmemBytes];
  float* xs = reinterpret_cast<float*>(smem + kStages * kStageBytes);                         // [rt][tt][32] x 4
  v4i* xc = reinterpret_cast<v4i*>(smem + kStages * kStageBytes + kXsBytes);                  // [rt][tt][64]
  float* xg = reinterpret_cast<float*>(smem + kStages * kStageBytes + kXsBytes + kXcBytes);   // [rt][32] x 4

  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const bool is_qk = w < 4;
  const int rt = (w & 3) >> 1, half = w & 1;     // QK: half = token tile; PV: half = dims half
  const int h = lane >> 5, n = lane & 31;

  // XCD-aware order: the row groups of one unit are 8 apart in launch order, so
  // they land on the same XCD and share its L2 for the KV pages.
  const int x8 = blockIdx.x & 7, q8i = blockIdx.x >> 3;
  const int g = q8i % a.G;
  const int unit = (q8i / a.G) * 8 + x8;
  const int units = a.chunk_blocks == 0 ? a.num_splits : a.B * a.num_splits;
  if (unit >= units) return;

  // ---- the global block range of this workgroup --------------------------
  int gstart, gend;
  if (a.chunk_blocks == 0) {
    const int64_t T = prefix[a.B];
    gstart = (int)((int64_t)unit * T / a.num_splits);
    gend = (int)((int64_t)(unit + 1) * T / a.num_splits);
  } else {
    const int b = unit / a.num_splits, s = unit % a.num_splits;
    const int nb = prefix[b + 1] - prefix[b];
    const int k0 = s * a.chunk_blocks;
    if (k0 >= nb) return;
    gstart = prefix[b] + k0;
    gend = prefix[b] + min(k0 + a.chunk_blocks, nb);
  }
  if (gstart >= gend) return;
  const int nblocks = gend - gstart;

  // ---- loader (every wave copies its share of each page) -------------------
  int ld_b = find_seq(prefix, a.B, gstart);
  int ld_gb = gstart;
  uint32_t stage_bad = 0;   // bit i: the page in stage i had an id out of range (wave-uniform)
  auto issue_next = [&](int stage_idx) {
    while (prefix[ld_b + 1] <= ld_gb) ++ld_b;
    const int blk = ld_gb - prefix[ld_b];
    int page = page_table[(int64_t)ld_b * a.max_pages + blk];
    const bool badp = page < 0 || page >= a.num_pages;
    if (badp) page = 0;
    stage_bad = (stage_bad & ~(1u << stage_idx)) | ((badp ? 1u : 0u) << stage_idx);
    const int valid = min(kPage, seq_lens[ld_b] - blk * kPage);
    issue_page(a.kv_latent, reinterpret_cast<const uint8_t*>(a.k_rope), a.kv_scale, a.zero, page, valid,
               smem + stage_idx * kStageBytes, w, lane);
    ++ld_gb;
  };
  issue_next(0);
  if (nblocks > 1) issue_next(1);

  const int row = 64 * g + 32 * rt + n;       // row of this lane within the sequence
  const bool row_ok = row < a.R;

  // piece bookkeeping (identical in every wave; scalar)
  int cur_b = -1, cur_blk0 = 0;
  bool cur_bad = false;
  auto piece_id = [&]() -> int64_t {
    return a.chunk_blocks == 0 ? (int64_t)unit + cur_b : (int64_t)cur_b * a.num_splits + cur_blk0 / a.chunk_blocks;
  };

  if (is_qk) {
    // ======================= QK / softmax waves ==============================
    const float sl2 = a.sl2;
    float cq = 0.f;                 // sigma_q * tau * log2(e)
    v8i qv[8];
    v4i qr[4];
    float m = -INFINITY, sp = 1.0f, l = 0.0f;
    int vis = 0;
    bool stored = false;

    auto write_lse = [&]() {
      if (half == 0 && h == 0 && row_ok) {
        float lse = l > 0.0f ? (m + log2f(sp * l)) * kLn2 : -INFINITY;
        if (cur_bad) lse = __builtin_nanf("");
        a.part_lse[piece_id() * a.rows_pad + row] = lse;
      }
    };

    for (int k = 0; k < nblocks; ++k) {
      block_barrier(stored || k + 1 >= nblocks);
      stored = false;
      const int gb = gstart + k;
      if (cur_b < 0 || gb >= prefix[cur_b + 1]) {        // first block of a new piece
        if (cur_b >= 0) { write_lse(); stored = true; }
        int b = cur_b < 0 ? find_seq(prefix, a.B, gb) : cur_b + 1;
        while (prefix[b + 1] <= gb) ++b;
        cur_b = b;
        cur_blk0 = gb - prefix[b];
        cur_bad = false;
        const int N = seq_lens[b];
        vis = a.causal ? N - a.q_len + 1 + row / a.H : N;
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
          cq = a.sq[qrow] * sl2;
        } else {
#pragma unroll
          for (int s = 0; s < 8; ++s) qv[s] = v8i{0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
          for (int s = 0; s < 4; ++s) qr[s] = v4i{0, 0, 0, 0};
          cq = 0.f;
        }
        m = -INFINITY; sp = 1.0f; l = 0.0f;
      }
      const int blk = gb - prefix[cur_b];
      cur_bad |= ((stage_bad >> (k % kStages)) & 1u) != 0;
      const uint8_t* st = smem + (k % kStages) * kStageBytes;

      // ---- S^T tile = K . Q^T ----------------------------------------------
      v16f accC = v16f{0}, accR = v16f{0};
      {
        const uint8_t* krow = st + (32 * half + n) * kDc;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          const v4i lo4 = *reinterpret_cast<const v4i*>(krow + (((4 * s + 2 * h) ^ n) << 4));
          const v4i hi4 = *reinterpret_cast<const v4i*>(krow + (((4 * s + 2 * h + 1) ^ n) << 4));
          const v8i A = v8i{lo4[0], lo4[1], lo4[2], lo4[3], hi4[0], hi4[1], hi4[2], hi4[3]};
          accC = mfma_f8_32x32x64(A, qv[s], accC);
        }
        const uint8_t* rrow = st + kLatBytes + (32 * half + n) * (kDr * 2);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const v4i A = *reinterpret_cast<const v4i*>(rrow + (((2 * s + h) ^ (n & 7)) << 4));
          accR = mfma_bf16_32x32x16(A, qr[s], accR);
        }
      }

      // ---- tile statistics: lane (row n, half h) holds tokens 32tt + 8(v/4) + 4h + v%4
      const float* st_sc = reinterpret_cast<const float*>(st + kLatBytes + kRopeBytes);
      float sk[16], pp[16];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const v4f f = *reinterpret_cast<const v4f*>(st_sc + 32 * half + 8 * q + 4 * h);
        sk[4 * q + 0] = f[0]; sk[4 * q + 1] = f[1]; sk[4 * q + 2] = f[2]; sk[4 * q + 3] = f[3];
      }
      const bool tail = (blk + 1) * kPage > vis;
      float mt = -INFINITY;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float x = accC[v] * (cq * sk[v]) + accR[v] * sl2;
        if (tail) {
          const int j = blk * kPage + 32 * half + 8 * (v >> 2) + 4 * h + (v & 3);
          x = j < vis ? x : -INFINITY;
        }
        pp[v] = x;
        mt = fmaxf(mt, x);
      }
      mt = xhalf_max(mt);                          // raw tile max of this row
      const float mloc = fmaxf(m, mt);             // reference of this tile's exponentials
      float esum = 0.f, pmax = 0.f;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float e = mloc > -INFINITY ? __builtin_amdgcn_exp2f(pp[v] - mloc) : 0.0f;
        esum += e;
        pp[v] = e * sk[v];
        pmax = fmaxf(pmax, pp[v]);
      }
      esum = xhalf_sum(esum);
      pmax = xhalf_max(pmax);
      if (h == 0) *reinterpret_cast<v4f*>(xs + ((rt * 2 + half) * 32 + n) * 4) = v4f{mt, esum, pmax, 0.f};
      barrier_vm_lgkm0<63>();
      if (k + 2 < nblocks) issue_next((k + 2) % kStages);

      // ---- block statistics, state update, probability codes --------------
      const v4f s0 = *reinterpret_cast<const v4f*>(xs + ((rt * 2 + 0) * 32 + n) * 4);
      const v4f s1 = *reinterpret_cast<const v4f*>(xs + ((rt * 2 + 1) * 32 + n) * 4);
      const float mb = fmaxf(s0[0], s1[0]);         // block max of the raw logits
      v4i mine = v4i{0, 0, 0, 0};
      float gam = 1.0f;
      if (mb > -INFINITY) {                         // the row sees a token of this block
        const float m_new = fmaxf(m, mb);
        const float a0 = __builtin_amdgcn_exp2f(fmaxf(m, s0[0]) - m_new);
        const float a1 = __builtin_amdgcn_exp2f(fmaxf(m, s1[0]) - m_new);
        const float lsum = a0 * s0[1] + a1 * s1[1];
        const float pbmax = fmaxf(a0 * s0[2], a1 * s1[2]);
        const float sP = fmaxf(pbmax / kFp8Max, kEps);
        const float inv = 1.0f / sP;
        gam = __builtin_amdgcn_exp2f(m - m_new) * (sp / sP);
        l = gam * l + lsum * inv;
        m = m_new;
        sp = sP;
        const float f = (half == 0 ? a0 : a1) * inv;
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          int wd = cvt_pk_e4m3(pp[4 * d + 0] * f, pp[4 * d + 1] * f, 0, false);
          wd = cvt_pk_e4m3(pp[4 * d + 2] * f, pp[4 * d + 3] * f, wd, true);
          mine[d] = wd;
        }
      }
      xc[(rt * 2 + half) * 64 + lane] = mine;
      if (half == 0 && h == 0) *reinterpret_cast<v4f*>(xg + (rt * 32 + n) * 4) = v4f{gam, l, 0.f, 0.f};
    }
    block_barrier(true);                           // pairs with the PV waves' last top barrier
    write_lse();
  } else {
    // =========================== PV waves ====================================
    v16f O[8];
#pragma unroll
    for (int T = 0; T < 8; ++T) O[T] = v16f{0};
    bool stored = false;

    // per-lane constant addressing of the transposed V reads: 16-lane group g16 of
    // half h reads 8 token rows x 16 bytes; lane pair (2i, 2i+1) supplies row i.
    const int q16 = lane & 15, tri = q16 >> 1, trb = q16 & 1, g16 = (lane >> 4) & 1;
    int tr_off[4], tr_x[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int tok = 16 * c + 8 * (tri >> 2) + 4 * h + (tri & 3);   // token of P/V slot 8c + tri
      tr_off[c] = tok * kDc + 8 * trb;
      tr_x[c] = tok & 31;
    }

    for (int k = 0; k <= nblocks; ++k) {
      block_barrier(stored || k + 1 >= nblocks);
      stored = false;
      if (k > 0) {
        // ---- PV of block k-1 with the codes the QK waves published ---------
        const uint8_t* st = smem + ((k - 1) % kStages) * kStageBytes;
        const v4f gl = *reinterpret_cast<const v4f*>(xg + (rt * 32 + n) * 4);
        const float gam = gl[0];
        const v4i c0 = xc[(rt * 2 + 0) * 64 + lane];
        const v4i c1 = xc[(rt * 2 + 1) * 64 + lane];
        const v8i P8 = v8i{c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
#pragma unroll
        for (int T = 0; T < 8; ++T) {
          const int chunk = 16 * half + 2 * T + g16;
          v2i r[4];
#pragma unroll
          for (int c = 0; c < 4; ++c) r[c] = lds_read_tr8(st + tr_off[c] + ((chunk ^ tr_x[c]) << 4));
          const v8i A = v8i{r[0][0], r[0][1], r[1][0], r[1][1], r[2][0], r[2][1], r[3][0], r[3][1]};
          O[T] = O[T] * gam;
          O[T] = mfma_f8_32x32x64(A, P8, O[T]);
        }
        // ---- end of a piece: write the normalized partial output ------------
        if (k == nblocks || gstart + k >= prefix[cur_b + 1]) {
          if (row_ok) {
            const float lfin = gl[1];
            const float inv = lfin > 0.0f ? 1.0f / lfin : 0.0f;
            const float nanv = __builtin_nanf("");
            float* po = a.part_o + (piece_id() * a.rows_pad + row) * kDc + 256 * half + 4 * h;
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
            stored = true;
          }
#pragma unroll
          for (int T = 0; T < 8; ++T) O[T] = v16f{0};
        }
      }
      if (k == nblocks) break;
      // piece bookkeeping for block k (mirrors the QK waves)
      const int gb = gstart + k;
      if (cur_b < 0 || gb >= prefix[cur_b + 1]) {
        int b = cur_b < 0 ? find_seq(prefix, a.B, gb) : cur_b + 1;
        while (prefix[b + 1] <= gb) ++b;
        cur_b = b;
        cur_blk0 = gb - prefix[b];
        cur_bad = false;
      }
      cur_bad |= ((stage_bad >> (k % kStages)) & 1u) != 0;
      barrier_vm_lgkm0<63>();
      if (k + 2 < nblocks) issue_next((k + 2) % kStages);
    }
  }
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream) {
  const int units = a.chunk_blocks == 0 ? a.num_splits : a.B * a.num_splits;
  if (units <= 0) return hipSuccess;
  const int64_t grid = (int64_t)((units + 7) / 8) * 8 * a.G;
  if (grid > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL(decode_kernel, dim3((unsigned)grid), dim3(64 * kWaves), 0, stream, a, a.prefix, a.page_table,
                     a.seq_lens);
  return hipGetLastError();
}

}  // namespace snapmla
