// FP8 MLA decode kernel (Algorithm 1; Appendix D recurrences; Section 3.2).
//
// One workgroup = 8 waves (two per SIMD) = 64 query rows of one row group x a
// contiguous range of 64-token KV blocks (one page each).  The waves specialise:
//   QK waves  w = 0..3, (rt, tt) = (w/2, w%2): S^T tile of row tile rt (32 rows)
//             and token tile tt (tokens 32tt..32tt+31), online softmax, scale
//             fusion and E4M3 probability codes; they own q and the row state.
//   PV waves  w = 4..7, (rt, dh) = ((w-4)/2, (w-4)%2): O^T of row tile rt and
//             latent dimensions 256dh..256dh+255; they own the output accumulator,
//             copy the pages into LDS and write the partial results.
// The two QK waves of a row tile exchange tile statistics through LDS and
// publish the probability codes and the per-row state; the PV waves consume
// them one block later.  So on every SIMD a QK wave works on block k while a PV
// wave works on block k-1, with two workgroup barriers per block.  (The paper's
// Hopper kernel splits the work between two warp groups, Algorithm 1 and
// Appendix E; here the split is by phase instead of by output half.)
//
// Data movement: each 64-token page (32 KiB E4M3 latent, 8 KiB bf16 RoPE,
// 256 B scales) is copied HBM -> LDS with 16-byte direct-to-LDS loads into a
// 3-stage ring, two pages ahead of the compute.  Latent rows are stored with the
// 16-byte chunk index XOR-swizzled by the token index (swz) so that both the
// token-major QK reads and the transposed PV reads avoid bank conflicts.  Page
// ids come from a 64-block window that one vector load fetches ahead of use.
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
// the monotone order of Appendix E.  Slots past the end of a sequence hold
// stale bytes; their logits are masked to -inf, their fused probabilities
// forced to 0 and their V bytes cleared before the PV product.

#include "snapmla_device.h"
#include "snapmla_internal.h"

namespace snapmla {

constexpr int kLatBytes = kPage * kDc;          // 32768
constexpr int kRopeBytes = kPage * kDr * 2;     // 8192
constexpr int kScBytes = kPage * 4;             // 256
constexpr int kStageBytes = kLatBytes + kRopeBytes + kScBytes;
constexpr int kStages = 3;
constexpr int kWaves = 8;
constexpr int kDmaPerBlock = 11;                // direct-to-LDS instructions per PV wave per page
constexpr int kXsBytes = 2 * 2 * 32 * 16;       // tile statistics [rt][tt][row] x float4
constexpr int kXcBytes = 2 * 2 * 64 * 16;       // probability codes [rt][tt][lane] x 16 B
constexpr int kXgBytes = 2 * 32 * 16;           // per-row gamma, l, m, sigma_p [rt][row] x float4
constexpr int kSmemBytes = kStages * kStageBytes + kXsBytes + kXcBytes + kXgBytes;
constexpr float kLn2 = 0.69314718055994531f;

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

  const int row = 64 * g + 32 * rt + n;       // row of this lane within the sequence
  const bool row_ok = row < a.R;

  // piece bookkeeping (identical in every wave; scalar)
  int cur_b = -1, cur_blk0 = 0, cur_end = 0, cur_n = 0;
  auto enter_piece = [&](int gb) {
    int b = cur_b < 0 ? find_seq(prefix, a.B, gb) : cur_b + 1;
    while (prefix[b + 1] <= gb) ++b;
    cur_b = b;
    cur_blk0 = gb - prefix[b];
    cur_end = prefix[b + 1];
    cur_n = seq_lens[b];
  };

  if (is_qk) {
    // ======================= QK / softmax waves ==============================
    const float sl2 = a.sl2;
    float cq = 0.f;                 // sigma_q * tau * log2(e)
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
    for (int s = 0; s < 4; ++s) roff[s] = kLatBytes + (32 * half + n) * (kDr * 2) + (((2 * s + h) ^ (n & 7)) << 4);
#pragma unroll
    for (int q = 0; q < 4; ++q) soff[q] = kLatBytes + kRopeBytes + 4 * (32 * half + 8 * q + 4 * h);

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
      const uint8_t* st = smem + (k % kStages) * kStageBytes;

      // ---- S^T tile = K . Q^T: operands of step s+1 load while step s multiplies
      v4f skq[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) skq[q] = *reinterpret_cast<const v4f*>(st + soff[q]);
      v16f accC = v16f{0}, accR = v16f{0};
      v4i c_lo = *reinterpret_cast<const v4i*>(st + koff[0]);
      v4i c_hi = *reinterpret_cast<const v4i*>(st + koff[1]);
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        v4i n_lo, n_hi;
        if (s < 7) {
          n_lo = *reinterpret_cast<const v4i*>(st + koff[2 * s + 2]);
          n_hi = *reinterpret_cast<const v4i*>(st + koff[2 * s + 3]);
        } else {
          n_lo = *reinterpret_cast<const v4i*>(st + roff[0]);
          n_hi = *reinterpret_cast<const v4i*>(st + roff[1]);
        }
        accC = mfma_f8_32x32x64(v8i{c_lo[0], c_lo[1], c_lo[2], c_lo[3], c_hi[0], c_hi[1], c_hi[2], c_hi[3]}, qv[s],
                                accC);
        c_lo = n_lo;
        c_hi = n_hi;
        __builtin_amdgcn_sched_barrier(0);
      }
      {
        const v4i r2 = *reinterpret_cast<const v4i*>(st + roff[2]);
        const v4i r3 = *reinterpret_cast<const v4i*>(st + roff[3]);
        accR = mfma_bf16_32x32x16(c_lo, qr[0], accR);
        accR = mfma_bf16_32x32x16(c_hi, qr[1], accR);
        accR = mfma_bf16_32x32x16(r2, qr[2], accR);
        accR = mfma_bf16_32x32x16(r3, qr[3], accR);
      }

      // ---- tile statistics: lane (row n, half h) holds tokens 32tt + 8(v/4) + 4h + v%4
      float sk[16], pp[16];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        sk[4 * q + 0] = skq[q][0]; sk[4 * q + 1] = skq[q][1]; sk[4 * q + 2] = skq[q][2]; sk[4 * q + 3] = skq[q][3];
      }
      const float rs = sl2;
#pragma unroll
      for (int v = 0; v < 16; ++v) pp[v] = fmaf(accC[v], cq * sk[v], accR[v] * rs);
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
      mt = xhalf_max(mt);                          // raw tile max of this row
      float mloc = fmaxf(m, mt);                   // reference of this tile's exponentials
      mloc = mloc > -INFINITY ? mloc : 0.0f;       // all -inf: exponentials become 0
      float e[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) e[v] = __builtin_amdgcn_exp2f(pp[v] - mloc);
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
      barrier_vm_lgkm0<63>();

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
      if (half == 0 && h == 0) *reinterpret_cast<v4f*>(xg + (rt * 32 + n) * 4) = v4f{gam, l, m, sp};
    }
    barrier_vm_lgkm0<63>();                        // pairs with the PV waves' last top barrier
  } else {
    // =========================== PV waves ====================================
    const int pw = __builtin_amdgcn_readfirstlane(w - 4);   // wave-uniform
    // constant per-lane byte offsets of this wave's share of a page copy
    uint32_t lat_off[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int P = 64 * (8 * pw + j) + lane;
      const int t = P >> 5, cp = P & 31;
      lat_off[j] = (uint32_t)(t * kDc + ((cp ^ swz(t)) << 4));
    }
    uint32_t rope_off[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int P = 64 * (2 * pw + j) + lane;
      const int t = P >> 3, cp = P & 7;
      rope_off[j] = (uint32_t)(t * (kDr * 2) + ((cp ^ (t & 7)) << 4));
    }
    const uint32_t sc_off = (uint32_t)((16 * pw + (lane & 15)) * 4);
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
    uint32_t stage_bad = 0;   // bit i: the page in stage i had an id out of range (wave-uniform)
    auto issue = [&](int kb, int page) {           // copy block gstart + kb into stage kb % 3
      const int stg = kb % kStages;
      const bool badp = page < 0 || page >= a.num_pages;
      if (badp) page = 0;
      stage_bad = (stage_bad & ~(1u << stg)) | ((badp ? 1u : 0u) << stg);
      const uint8_t* lat = a.kv_latent + (int64_t)page * kLatBytes;
      const uint8_t* rp = reinterpret_cast<const uint8_t*>(a.k_rope) + (int64_t)page * kRopeBytes;
      const uint8_t* sc = reinterpret_cast<const uint8_t*>(a.kv_scale) + (int64_t)page * kScBytes;
      const uint32_t sb = smem_base + stg * kStageBytes;
#pragma unroll
      for (int i = 0; i < 8; ++i) g2lds16_so(lat, lat_off[i], sb + 1024 * (8 * pw + i));
#pragma unroll
      for (int i = 0; i < 2; ++i) g2lds16_so(rp, rope_off[i], sb + kLatBytes + 1024 * (2 * pw + i));
      if (lane < 16) g2lds4_so(sc, sc_off, sb + kLatBytes + kRopeBytes + 64 * pw);
    };
    issue(0, page_of(0));
    if (nblocks > 1) issue(1, page_of(1));

    v16f O[8];
#pragma unroll
    for (int T = 0; T < 8; ++T) O[T] = v16f{0};
    bool stored = false, cur_bad = false;

    // transposed V reads: 16-lane group g16 of half h reads 8 token rows x 16 bytes;
    // lane pair (2i, 2i+1) supplies row i (token of P/V slot 8c + i).  The byte
    // offset of tile T, read c inside a stage is tr_base[c] + (tr_y[c] ^ (T << 5)):
    // the swizzled chunk index is ((16 half + g16) ^ tok) ^ 2T.
    const int q16 = lane & 15, tri = q16 >> 1, trb = q16 & 1, g16 = (lane >> 4) & 1;
    uint32_t tr_base[4], tr_y[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int tok = 16 * c + 8 * (tri >> 2) + 4 * h + (tri & 3);
      tr_base[c] = tok * kDc + 8 * trb;
      tr_y[c] = (uint32_t)(((16 * half + g16) ^ swz(tok)) << 4);
    }
    int prev_valid = kPage;                        // valid tokens of the pending block

    for (int k = 0; k <= nblocks; ++k) {
      if (stored || k + 1 >= nblocks) barrier_vm_lgkm0<0>(); else barrier_vm_lgkm0<kDmaPerBlock>();
      stored = false;
      // page id of the block copied after the mid-period barrier (scalar load,
      // in flight during the PV product)
      const int pg2 = k + 2 < nblocks ? page_of(k + 2) : 0;
      if (k > 0) {
        // ---- PV of block k-1 with the codes the QK waves published ---------
        const uint8_t* st = smem + ((k - 1) % kStages) * kStageBytes;
        const uint8_t* trp[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) trp[c] = st + tr_base[c];
        const v4f gl = *reinterpret_cast<const v4f*>(xg + (rt * 32 + n) * 4);
        const float gam = gl[0];
        const v4i c0 = xc[(rt * 2 + 0) * 64 + lane];
        const v4i c1 = xc[(rt * 2 + 1) * 64 + lane];
        const v8i P8 = v8i{c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
        if (prev_valid < kPage) {
          // last page of a sequence: clear the bytes of the slots past its end that
          // this wave reads (stale data could hold NaN codes; their probability
          // codes are 0).  The other wave of this dims half writes the same zeros.
          const int nz = (kPage - prev_valid) * 16;
          for (int i = lane; i < nz; i += 64) {
            const int t = prev_valid + (i >> 4);
            const int c = 16 * half + (i & 15);
            *reinterpret_cast<v4i*>(const_cast<uint8_t*>(st) + t * kDc + ((c ^ swz(t)) << 4)) = v4i{0, 0, 0, 0};
          }
        }
        v2i rc[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) rc[c] = lds_read_tr8(trp[c] + tr_y[c]);
#pragma unroll
        for (int T = 0; T < 8; ++T) {
          v2i rn[4];
          if (T < 7) {
#pragma unroll
            for (int c = 0; c < 4; ++c) rn[c] = lds_read_tr8(trp[c] + (tr_y[c] ^ opaque_u32((T + 1) << 5)));
          }
          const v8i A = v8i{rc[0][0], rc[0][1], rc[1][0], rc[1][1], rc[2][0], rc[2][1], rc[3][0], rc[3][1]};
          O[T] = O[T] * gam;
          O[T] = mfma_f8_32x32x64(A, P8, O[T]);
          if (T < 7) {
#pragma unroll
            for (int c = 0; c < 4; ++c) rc[c] = rn[c];
          }
          __builtin_amdgcn_sched_barrier(0);
        }
        // ---- end of a piece: write the normalized partial output and LSE ----
        if (k == nblocks || gstart + k >= cur_end) {
          if (row_ok) {
            const float lfin = gl[1];
            const bool empty = !(lfin > 0.0f);
            const float inv = empty ? 0.0f : 1.0f / lfin;
            const float nanv = __builtin_nanf("");
            const int64_t pid = a.chunk_blocks == 0 ? (int64_t)unit + cur_b
                                                    : (int64_t)cur_b * a.num_splits + cur_blk0 / a.chunk_blocks;
            float* po = a.part_o + (pid * a.rows_pad + row) * kDc + 256 * half + 4 * h;
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
            if (half == 0 && h == 0) {
              float lse = empty ? -INFINITY : (gl[2] + log2f(gl[3] * lfin)) * kLn2;
              if (cur_bad) lse = nanv;
              a.part_lse[pid * a.rows_pad + row] = lse;
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
      if (cur_b < 0 || gb >= cur_end) {
        enter_piece(gb);
        cur_bad = false;
      }
      cur_bad |= ((stage_bad >> (k % kStages)) & 1u) != 0;
      prev_valid = min(kPage, cur_n - (gb - prefix[cur_b]) * kPage);
      barrier_vm_lgkm0<63>();
      if (k + 2 < nblocks) issue(k + 2, pg2);
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
