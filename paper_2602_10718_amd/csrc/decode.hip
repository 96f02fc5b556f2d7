// FP8 MLA decode kernel (Algorithm 1; Appendix D recurrences; Section 3.2).
//
// One workgroup = 8 waves (two per SIMD) = 64 query rows of one row group x a
// contiguous range of 64-token KV blocks (one page each).  The waves specialise:
//   QK waves  w = 0..3, (rt, tt) = (w/2, w%2): S^T tile of row tile rt (32 rows)
//             and token tile tt (tokens 32tt..32tt+31), online softmax, scale
//             fusion and E4M3 probability codes; they own q and the row state.
//   PV waves  w = 4..7, dq = w-4: O^T of all 64 rows for latent dimensions
//             128dq..128dq+127 (each V^T tile read from LDS once, used for both
//             row tiles); they own the output accumulator, copy the pages into
//             LDS and write the partial results.
// The two QK waves of a row tile exchange tile statistics through LDS with a
// flag handshake of their own, then publish the probability codes and the
// per-row state; the PV waves consume them one block later.  So on every SIMD a
// QK wave works on block k while a PV wave works on block k-1, with one
// workgroup barrier per block.  The code/state buffers are single: a QK wave
// overwrites them only after every PV wave has flagged that it holds the
// previous block's values in registers.  (The paper's Hopper kernel splits the
// work between two warp groups, Algorithm 1 and Appendix E; here the split is by
// phase instead of by output half.)
//
// Data movement: each 64-token page (32 KiB E4M3 latent, 8 KiB bf16 RoPE,
// 256 B scales) is copied HBM -> LDS with 16-byte direct-to-LDS loads, two
// pages ahead of the compute, right after the barrier that opens a period, so
// every page has two full periods to arrive.  The latent lives four periods in
// LDS (arriving, arriving, QK, PV) and the RoPE/scale part three (it is only
// read by the QK waves), hence a 4-stage latent ring and a 3-stage RoPE/scale
// ring (160 KiB of LDS in all).  Latent rows are stored with the 16-byte chunk
// index XOR-swizzled by the token index (swz) so that both the token-major QK
// reads and the transposed PV reads avoid bank conflicts.  Page ids are read
// with scalar loads one block ahead of their copy.
//
// Per block (matrices transposed so that one lane owns one query row):
//   S^T[32 tok x 32 rows]  = K_c^T . q8^T   (32x32x64 FP8 MFMA, K = 512)
//                          + K_r^T . q_r^T  (32x32x16 BF16 MFMA, K = 64)
//   s = log2(e) tau (sigma_q sigma_K acc_c + acc_r)   (Section 3.1 domain alignment,
//       applied to the two accumulators instead of pre-scaling the RoPE operands)
//   running max m, block scale sigma_P = max(max(e sigma_K) / 448, 2^-40),
//   gamma = exp(m_old - m) sigma_p_old / sigma_P, l = gamma l + sum(e) / sigma_P,
//   codes pi = E4M3(e sigma_K / sigma_P)                 (Appendix D)
//   O^T[128 dims x 64 rows] = gamma O^T + V^T . P^T       (FP8 MFMA, K = 64 tokens)
// V^T is read straight from the token-major latent tile with the LDS transpose
// read (ds_read_b64_tr_b8; the CDNA counterpart of the paper's V-tile
// transposition) and the P codes are already in the B-operand layout, so no
// accumulator permutation is needed.  Blocks are consumed in increasing order,
// the monotone order of Appendix E.  Slots past the end of a sequence hold
// stale bytes; their logits are masked to -inf, their fused probabilities
// forced to 0 and their V bytes cleared before the PV product.

#include "snapmla_device.h"
#include "snapmla_internal.h"

namespace snapmla {

constexpr int kLatBytes = kPage * kDc;          // 32768
constexpr int kRopeBytes = kPage * kDr * 2;     // 8192
constexpr int kScBytes = kPage * 4;             // 256
constexpr int kRsBytes = kRopeBytes + kScBytes;  // RoPE + scale part of a page
constexpr int kLatStages = 4;
constexpr int kRsStages = 3;
constexpr int kRsBase = kLatStages * kLatBytes;   // LDS offset of the RoPE/scale ring
constexpr int kXBase = kRsBase + kRsStages * kRsBytes;
constexpr int kWaves = 8;
constexpr int kXsBytes = 2 * 2 * 32 * 16;       // tile statistics [rt][tt][row] x float4
constexpr int kXcBytes = 2 * 2 * 64 * 16;       // probability codes [rt][tt][lane] x 16 B
constexpr int kXgBytes = 2 * 32 * 16;           // per-row gamma, l, m, sigma_p [rt][row] x float4
constexpr int kXfBytes = 8 * 4;                 // handshake flags: [QK wave], [PV wave]
constexpr int kSmemBytes = kXBase + kXsBytes + kXcBytes + kXgBytes + kXfBytes;
static_assert(kSmemBytes <= 160 * 1024, "LDS budget of one workgroup");
constexpr float kLn2 = 0.69314718055994531f;
// Upper bound on the polls of a handshake wait.  The waits end by construction
// (every flag they poll is stored once per block, before its owner waits on
// anything); the bound only guarantees that the kernel terminates.
constexpr int kSpinLimit = 1 << 22;

// Latent rows are stored with 16-byte chunk c of token t at chunk c ^ swz(t).
// Eight consecutive tokens (token-major QK reads) and the eight tokens
// {t0..t0+3, t0+8..t0+11} of one transposed-read group (PV reads) both map a
// given chunk to eight distinct 128-byte bank lines.
__device__ __forceinline__ int swz(int t) { return (t & 31) ^ (((t >> 3) & 1) << 2); }

// Largest b with prefix[b] <= gb (prefix is non-decreasing, prefix[B] > gb).
__device__ __forceinline__ int find_seq(const int32_t* __restrict__ prefix, int B, int gb) {
  int lo = 0, hi = B - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (prefix[mid] <= gb) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Handshake flags in LDS.  A wave's LDS operations complete in issue order, so
// a flag stored after lds_wait_all() is seen only after the data stored before it.
__device__ __forceinline__ void lds_wait_all() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
__device__ __forceinline__ void flag_store(int* f, int v) {
  __hip_atomic_store(f, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ int flag_load(const int* f) {
  return __hip_atomic_load(const_cast<int*>(f), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
// Four consecutive flags with one LDS read (an explicit LDS pointer: a generic one
// would become a flat load, which queues behind the page copies).
typedef __attribute__((address_space(3))) volatile v4i lds_flags4;
__device__ __forceinline__ v4i flag_load4(const int* f) { return *(const lds_flags4*)(f); }

__global__ __launch_bounds__(512, 1) void decode_kernel(DecodeArgs a, const int32_t* __restrict__ prefix,
                                                        const int32_t* __restrict__ page_table,
                                                        const int32_t* __restrict__ seq_lens) {
  __shared__ __attribute__((aligned(1024))) uint8_t smem[kSmemBytes];
  float* xs = reinterpret_cast<float*>(smem + kXBase);                          // [rt][tt][32] x 4
  v4i* xc = reinterpret_cast<v4i*>(smem + kXBase + kXsBytes);                   // [rt][tt][64]
  float* xg = reinterpret_cast<float*>(smem + kXBase + kXsBytes + kXcBytes);    // [64 rows] x 4
  int* xf = reinterpret_cast<int*>(smem + kXBase + kXsBytes + kXcBytes + kXgBytes);   // [0..3] QK, [4..7] PV

  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const bool is_qk = w < 4;
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

  // piece bookkeeping (identical in every wave; scalar)
  int cur_b = -1, cur_blk0 = 0, cur_end = 0, cur_n = 0, cur_p0 = 0;
  auto enter_piece = [&](int gb) {
    int b = cur_b < 0 ? find_seq(prefix, a.B, gb) : cur_b + 1;
    while (prefix[b + 1] <= gb) ++b;
    cur_b = b;
    cur_p0 = prefix[b];
    cur_blk0 = gb - cur_p0;
    cur_end = prefix[b + 1];
    cur_n = seq_lens[b];
  };

  if (lane == 0) flag_store(xf + w, 0);            // ordered before any wait by the first barrier

  if (is_qk) {
    // ======================= QK / softmax waves ==============================
    const int rt = w >> 1, half = w & 1;           // half = token tile
    const int row = 64 * g + 32 * rt + n;          // query row of this lane within the sequence
    const bool row_ok = row < a.R;
    const float sl2 = a.sl2;
    float cq = 0.f;                 // sigma_q
    v8i qv[8];
    v4i qr[4];
    float m = -INFINITY, sp = 1.0f, l = 0.0f;
    int vis = 0;
    // per-lane LDS byte offsets inside a stage (constant across blocks): the 16
    // latent chunks of this lane's token for the 8 K-steps, its 4 RoPE chunks and
    // the scales of its 16 tokens (4 x float4)
    uint32_t koff[16], roff[4], soff[4];
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      koff[2 * s] = (32 * half + n) * kDc + (((4 * s + 2 * h) ^ swz(n)) << 4);
      koff[2 * s + 1] = (32 * half + n) * kDc + (((4 * s + 2 * h + 1) ^ swz(n)) << 4);
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) roff[s] = (32 * half + n) * (kDr * 2) + (((2 * s + h) ^ (n & 7)) << 4);
#pragma unroll
    for (int q = 0; q < 4; ++q) soff[q] = kRopeBytes + 4 * (32 * half + 8 * q + 4 * h);

    for (int k = 0; k < nblocks; ++k) {
      barrier_vm_lgkm0<63>();                              // page k has landed (PV waves waited)
      const int gb = gstart + k;
      if (cur_b < 0 || gb >= cur_end) {                    // first block of a new piece
        enter_piece(gb);
        vis = a.causal ? cur_n - a.q_len + 1 + row / a.H : cur_n;
        if (row_ok) {
          const int64_t qrow = (int64_t)cur_b * a.R + row;
          const v4i* src = reinterpret_cast<const v4i*>(a.q8 + qrow * kDc);
#pragma unroll
          for (int s = 0; s < 8; ++s) {
            const v4i lo4 = src[4 * s + 2 * h], hi4 = src[4 * s + 2 * h + 1];
            qv[s] = v8i{lo4[0], lo4[1], lo4[2], lo4[3], hi4[0], hi4[1], hi4[2], hi4[3]};
          }
          const v4i* rsrc = reinterpret_cast<const v4i*>(a.q_rope + qrow * kDr);
#pragma unroll
          for (int s = 0; s < 4; ++s) qr[s] = rsrc[2 * s + h];
          cq = a.sq[qrow];
        } else {
#pragma unroll
          for (int s = 0; s < 8; ++s) qv[s] = v8i{0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
          for (int s = 0; s < 4; ++s) qr[s] = v4i{0, 0, 0, 0};
          cq = 0.f;
        }
        m = -INFINITY; sp = 1.0f; l = 0.0f;
      }
      const int blk = gb - cur_p0;
      const uint8_t* st = smem + (k % kLatStages) * kLatBytes;             // latent of block k
      const uint8_t* sr = smem + kRsBase + (k % kRsStages) * kRsBytes;     // its RoPE and scales

      // ---- S^T tile = K . Q^T: every operand of the block is requested before the
      // first product, so the LDS latency is paid once per block
      v4f skq[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) skq[q] = *reinterpret_cast<const v4f*>(sr + soff[q]);
      v4i kc[16], kr[4];
#pragma unroll
      for (int i = 0; i < 16; ++i) kc[i] = *reinterpret_cast<const v4i*>(st + koff[i]);
#pragma unroll
      for (int i = 0; i < 4; ++i) kr[i] = *reinterpret_cast<const v4i*>(sr + roff[i]);
      __builtin_amdgcn_sched_barrier(0);           // keep the reads ahead of the products
      v16f accC = v16f{0}, accR = v16f{0};
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        accC = mfma_f8_32x32x64(v8i{kc[2 * s][0], kc[2 * s][1], kc[2 * s][2], kc[2 * s][3], kc[2 * s + 1][0],
                                    kc[2 * s + 1][1], kc[2 * s + 1][2], kc[2 * s + 1][3]},
                                qv[s], accC);
        if (s < 4) accR = mfma_bf16_32x32x16(kr[s], qr[s], accR);
      }

      // ---- tile statistics: lane (row n, half h) holds tokens 32tt + 8(v/4) + 4h + v%4
      float sk[16], pp[16];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        sk[4 * q + 0] = skq[q][0]; sk[4 * q + 1] = skq[q][1]; sk[4 * q + 2] = skq[q][2]; sk[4 * q + 3] = skq[q][3];
      }
      // raw logits u = sigma_q sigma_K acc_c + acc_r; s = tau log2(e) u enters the
      // exponentials through one fma each
#pragma unroll
      for (int v = 0; v < 16; ++v) pp[v] = fmaf(accC[v], cq * sk[v], accR[v]);
      const bool tail = (blk + 1) * kPage > vis;   // some token of this block is hidden from this row
      if (tail) {
        // hidden tokens and stale slots past the sequence end: logit -inf
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int j = blk * kPage + 32 * half + 8 * (v >> 2) + 4 * h + (v & 3);
          pp[v] = j < vis ? pp[v] : -INFINITY;
        }
      }
      float mt = fmaxf(fmaxf(fmaxf(pp[0], pp[1]), fmaxf(pp[2], pp[3])), fmaxf(fmaxf(pp[4], pp[5]), fmaxf(pp[6], pp[7])));
      mt = fmaxf(mt, fmaxf(fmaxf(fmaxf(pp[8], pp[9]), fmaxf(pp[10], pp[11])),
                           fmaxf(fmaxf(pp[12], pp[13]), fmaxf(pp[14], pp[15]))));
      mt = xhalf_max(mt) * sl2;                    // tile max of this row (log2 units)
      float mloc = fmaxf(m, mt);                   // reference of this tile's exponentials
      mloc = mloc > -INFINITY ? mloc : 0.0f;       // all -inf: exponentials become 0
      float e[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) e[v] = __builtin_amdgcn_exp2f(fmaf(pp[v], sl2, -mloc));
      if (tail) {
#pragma unroll
        for (int v = 0; v < 16; ++v) sk[v] = pp[v] > -INFINITY ? sk[v] : 0.0f;   // stale scales may be NaN
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) pp[v] = e[v] * sk[v];
      float esum = ((e[0] + e[1]) + (e[2] + e[3])) + ((e[4] + e[5]) + (e[6] + e[7]));
      esum += ((e[8] + e[9]) + (e[10] + e[11])) + ((e[12] + e[13]) + (e[14] + e[15]));
      float pmax = fmaxf(fmaxf(fmaxf(pp[0], pp[1]), fmaxf(pp[2], pp[3])), fmaxf(fmaxf(pp[4], pp[5]), fmaxf(pp[6], pp[7])));
      pmax = fmaxf(pmax, fmaxf(fmaxf(fmaxf(pp[8], pp[9]), fmaxf(pp[10], pp[11])),
                               fmaxf(fmaxf(pp[12], pp[13]), fmaxf(pp[14], pp[15]))));
      esum = xhalf_sum(esum);
      pmax = xhalf_max(pmax);
      if (h == 0) *reinterpret_cast<v4f*>(xs + ((rt * 2 + half) * 32 + n) * 4) = v4f{mt, esum, pmax, 0.f};
      // handshake with the other QK wave of this row tile: publish, then wait
      // for its statistics of the same block (it never waits on anything else
      // before publishing, so the wait ends)
      lds_wait_all();
      if (lane == 0) flag_store(xf + w, k + 1);
      for (int spin = 0; spin < kSpinLimit && flag_load(xf + (w ^ 1)) != k + 1; ++spin) {
      }
      asm volatile("" ::: "memory");

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
        // (reciprocals instead of divisions: off by at most an ulp, far inside the
        // rounding slack of the probability codes)
        const float sP = fmaxf(pbmax * (1.0f / kFp8Max), kEps);
        const float inv = __builtin_amdgcn_rcpf(sP);
        gam = __builtin_amdgcn_exp2f(m - m_new) * (sp * inv);
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
      // the PV waves hold block k-1's codes and state once all four flagged k
      if (k > 0) {
        for (int spin = 0; spin < kSpinLimit; ++spin) {
          const v4i f4 = flag_load4(xf + 4);
          if (f4[0] >= k && f4[1] >= k && f4[2] >= k && f4[3] >= k) break;
        }
        asm volatile("" ::: "memory");
      }
      xc[(rt * 2 + half) * 64 + lane] = mine;
      if (half == 0 && h == 0) *reinterpret_cast<v4f*>(xg + (32 * rt + n) * 4) = v4f{gam, l, m, sp};
    }
    barrier_vm_lgkm0<63>();                        // pairs with the PV waves' last top barrier
  } else {
    // =========================== PV waves ====================================
    const int dq = __builtin_amdgcn_readfirstlane(w - 4);   // dims 128dq..128dq+127; wave-uniform
    const int row0 = 64 * g + n, row1 = row0 + 32;          // query rows of this lane (row tiles 0, 1)
    // This wave copies latent rows 16dq..16dq+15 (instruction j: rows 16dq + 2j + h,
    // LDS chunk n of the row takes global chunk n ^ swz(row)), RoPE rows
    // 16dq..16dq+15 and scales 16dq..16dq+15 of each page.  For row t = 16dq + 2j + h,
    // n ^ swz(t) = (n ^ h) ^ cj with the wave-uniform cj = (16(dq&1) + 2j) ^ (j >= 4 ? 4 : 0),
    // so one per-lane register serves all eight latent copies:
    //   global offset = (16dq + 2j) * 512 + (lat_v ^ (cj << 4)).
    const uint32_t lat_v = (uint32_t)((((n ^ h) << 4)) | (h << 9));
    // RoPE instruction j covers rows 16dq + 8j + lane/8, chunk lane%8 ^ (lane/8)
    const uint32_t rope_v = (uint32_t)((lane >> 3) * (kDr * 2) + (((lane & 7) ^ (lane >> 3)) << 4));
    const uint32_t sc_off = (uint32_t)((16 * dq + (lane & 15)) * 4);
    const uint32_t smem_base = lds_offset(smem);

    // issue cursor (scalar): the next block to copy lies in sequence ib, whose
    // blocks are global blocks [ib_lo, ib_hi).  Blocks are requested in order.
    int ib = find_seq(prefix, a.B, gstart);
    int ib_lo = prefix[ib], ib_hi = prefix[ib + 1];
    auto page_of = [&](int kb) -> int {
      const int gb = gstart + kb;
      while (gb >= ib_hi) {                        // skips sequences without blocks
        ++ib;
        ib_lo = ib_hi;
        ib_hi = prefix[ib + 1];
      }
      return page_table[(int64_t)ib * a.max_pages + (gb - ib_lo)];
    };
    // Copies per PV wave and page: 8 latent instructions, then 2 RoPE + 1 scale
    // instruction, addressed by a wave-uniform base and the per-lane offsets above.
    // Block j is copied right after the barrier that opens period j-2: its latent
    // stage held block j-4 (PV product done in period j-3) and its RoPE/scale stage
    // block j-3 (read by the QK waves in period j-3).
    uint32_t stage_bad = 0;   // bit i: the page in latent stage i had an id out of range (wave-uniform)
    auto page_ok = [&](int page) { return page >= 0 && page < a.num_pages; };
    auto copy_latent = [&](int kb, int page) {
      const int stg = kb % kLatStages;
      const bool badp = !page_ok(page);
      if (badp) page = 0;
      stage_bad = (stage_bad & ~(1u << stg)) | ((badp ? 1u : 0u) << stg);
      const uint8_t* src = a.kv_latent + (int64_t)page * kLatBytes;
      const uint32_t dst = smem_base + stg * kLatBytes;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t cj = (uint32_t)(((16 * (dq & 1) + 2 * i) ^ (i >= 4 ? 4 : 0)) << 4);
        g2lds16_so(src + (16 * dq + 2 * i) * kDc, lat_v ^ cj, dst + 1024 * (8 * dq + i));
      }
    };
    auto copy_rope_scale = [&](int kb, int page) {
      if (!page_ok(page)) page = 0;
      const uint8_t* rp = reinterpret_cast<const uint8_t*>(a.k_rope) + (int64_t)page * kRopeBytes;
      const uint8_t* sc = reinterpret_cast<const uint8_t*>(a.kv_scale) + (int64_t)page * kScBytes;
      const uint32_t dst = smem_base + kRsBase + (kb % kRsStages) * kRsBytes;
#pragma unroll
      for (int i = 0; i < 2; ++i) g2lds16_so(rp + (16 * dq + 8 * i) * (kDr * 2), rope_v, dst + 1024 * (2 * dq + i));
      if (lane < 16) g2lds4_so(sc, sc_off, dst + kRopeBytes + 64 * dq);
    };
    // prologue: blocks 0 and 1
    const int pg0 = page_of(0);
    copy_latent(0, pg0);
    copy_rope_scale(0, pg0);
    if (nblocks > 1) {
      const int pg1 = page_of(1);
      copy_latent(1, pg1);
      copy_rope_scale(1, pg1);
    }
    int pg_n = nblocks > 2 ? page_of(2) : 0;       // page id of block k+2 in period k

    // O[2T + r]: O^T tile of dims 128dq + 32T.. and row tile r
    v16f O[8];
#pragma unroll
    for (int T = 0; T < 8; ++T) O[T] = v16f{0};
    bool cur_bad = false;

    // transposed V reads: 16-lane group g16 of half h reads 8 token rows x 16 bytes;
    // lane pair (2i, 2i+1) supplies row i (token of P/V slot 8c + i).  The byte
    // offset of tile T, read c inside a stage is tr_off[c] ^ (T << 5): the row
    // offset, byte half and swizzled chunk ((8dq + g16) ^ swz(tok)) ^ 2T occupy
    // disjoint bits, and so does the stage base.
    const int q16 = lane & 15, tri = q16 >> 1, trb = q16 & 1, g16 = (lane >> 4) & 1;
    uint32_t tr_off[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int tok = 16 * c + 8 * (tri >> 2) + 4 * h + (tri & 3);
      tr_off[c] = (uint32_t)(tok * kDc + 8 * trb) | (uint32_t)(((8 * dq + g16) ^ swz(tok)) << 4);
    }
    // Top-of-period wait: block k complete, block k+1 (11 copies) may stay in
    // flight.  Loads complete in issue order, so "at most 11 outstanding" implies
    // block k is in LDS even with the previous period's stores still counted.
    auto top_barrier = [&](int k) {
      if (k + 1 >= nblocks) barrier_vm_lgkm0<0>();
      else barrier_vm_lgkm0<11>();
    };

    // period 0: no PV product yet
    top_barrier(0);
    if (nblocks > 2) {
      copy_latent(2, pg_n);
      copy_rope_scale(2, pg_n);
      if (nblocks > 3) pg_n = page_of(3);
    }
    enter_piece(gstart);
    cur_bad = (stage_bad & 1u) != 0;
    int prev_valid = min(kPage, cur_n - (gstart - cur_p0) * kPage);   // valid tokens of the pending block

    for (int k = 1; k <= nblocks; ++k) {
      top_barrier(k);
      const bool copy = k + 2 < nblocks;
      if (copy) {
        copy_latent(k + 2, pg_n);
        copy_rope_scale(k + 2, pg_n);
      }
      // ---- PV of block k-1 with the codes the QK waves published -----------
      const uint32_t st_lds = smem_base + ((k - 1) % kLatStages) * kLatBytes;
      const v4f gl0 = *reinterpret_cast<const v4f*>(xg + n * 4);
      const v4f gl1 = *reinterpret_cast<const v4f*>(xg + (n + 32) * 4);
      const v4i c00 = xc[0 * 64 + lane], c01 = xc[1 * 64 + lane];
      const v4i c10 = xc[2 * 64 + lane], c11 = xc[3 * 64 + lane];
      const v8i P0 = v8i{c00[0], c00[1], c00[2], c00[3], c01[0], c01[1], c01[2], c01[3]};
      const v8i P1 = v8i{c10[0], c10[1], c10[2], c10[3], c11[0], c11[1], c11[2], c11[3]};
      const float gam0 = gl0[0], gam1 = gl1[0];
      // codes and state are in registers: let the QK waves overwrite them
      lds_wait_all();
      if (lane == 0) flag_store(xf + w, k);
      if (k + 3 < nblocks) pg_n = page_of(k + 3);    // scalar load, in flight during the product
      if (prev_valid < kPage) {
        // last page of a sequence: clear the bytes of the slots past its end that
        // this wave reads (stale data could hold NaN codes; their probability
        // codes are 0)
        uint8_t* stp = smem + ((k - 1) % kLatStages) * kLatBytes;
        const int nz = (kPage - prev_valid) * 8;
        for (int i = lane; i < nz; i += 64) {
          const int t = prev_valid + (i >> 3);
          const int c = 8 * dq + (i & 7);
          *reinterpret_cast<v4i*>(stp + t * kDc + ((c ^ swz(t)) << 4)) = v4i{0, 0, 0, 0};
        }
      }
      // all 16 transposed reads first, then the rescale, then the 8 products
      v2i rv[4][4];
#pragma unroll
      for (int T = 0; T < 4; ++T) {
#pragma unroll
        for (int c = 0; c < 4; ++c) rv[T][c] = lds_read_tr8_at((st_lds | tr_off[c]) ^ (uint32_t)(T << 5));
      }
#pragma unroll
      for (int T = 0; T < 4; ++T) {
        O[2 * T] *= gam0;
        O[2 * T + 1] *= gam1;
      }
#pragma unroll
      for (int T = 0; T < 4; ++T) {
        const v8i A = v8i{rv[T][0][0], rv[T][0][1], rv[T][1][0], rv[T][1][1],
                          rv[T][2][0], rv[T][2][1], rv[T][3][0], rv[T][3][1]};
        O[2 * T] = mfma_f8_32x32x64(A, P0, O[2 * T]);
        O[2 * T + 1] = mfma_f8_32x32x64(A, P1, O[2 * T + 1]);
      }
      // ---- end of a piece: write the normalized partial output and LSE ------
      // (one 16-byte store at a time; a bad page id makes the multiplier NaN)
      if (k == nblocks || gstart + k >= cur_end) {
        const int64_t pid = a.chunk_blocks == 0 ? (int64_t)unit + cur_b
                                                : (int64_t)cur_b * a.num_splits + cur_blk0 / a.chunk_blocks;
        const float nanv = __builtin_nanf("");
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          const int row = r == 0 ? row0 : row1;
          if (row < a.R) {
            const v4f gl = r == 0 ? gl0 : gl1;
            const float lfin = gl[1];
            const bool empty = !(lfin > 0.0f);
            float inv = empty ? 0.0f : 1.0f / lfin;
            if (cur_bad) inv = nanv;
            float* po = a.part_o + (pid * a.rows_pad + row) * kDc + 128 * dq + 4 * h;
#pragma unroll
            for (int T = 0; T < 4; ++T) {
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                *reinterpret_cast<v4f*>(po + 32 * T + 8 * q) =
                    v4f{O[2 * T + r][4 * q + 0] * inv, O[2 * T + r][4 * q + 1] * inv,
                        O[2 * T + r][4 * q + 2] * inv, O[2 * T + r][4 * q + 3] * inv};
                __builtin_amdgcn_sched_barrier(0);
              }
            }
            if (dq == 0 && h == 0) {
              float lse = empty ? -INFINITY : (gl[2] + log2f(gl[3] * lfin)) * kLn2;
              if (cur_bad) lse = nanv;
              a.part_lse[pid * a.rows_pad + row] = lse;
            }
          }
        }
#pragma unroll
        for (int T = 0; T < 8; ++T) O[T] = v16f{0};
      }
      if (k == nblocks) break;
      // piece bookkeeping for block k (mirrors the QK waves)
      const int gb = gstart + k;
      if (gb >= cur_end) {
        enter_piece(gb);
        cur_bad = false;
      }
      cur_bad |= ((stage_bad >> (k % kLatStages)) & 1u) != 0;
      prev_valid = min(kPage, cur_n - (gb - cur_p0) * kPage);
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
