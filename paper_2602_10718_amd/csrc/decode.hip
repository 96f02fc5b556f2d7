// FP8 MLA decode kernel (Algorithm 1; Appendix D recurrences; Section 3.2).
//
// One workgroup = 8 waves (two per SIMD) = 64 query rows of one row group x a
// contiguous range of 64-token KV blocks (one page each).  The waves specialise:
//   QK waves  w = 0..3: rows 16w..16w+15 against all 64 tokens of a block
//             (16x16 tiles, tokens on the MFMA M axis, so one lane holds 16
//             logits of one row and the four lanes of a row complete the block);
//             online softmax, scale fusion and E4M3 probability codes; they own
//             q and the row state.
//   PV waves  w = 4..7, dq = w-4: O^T of all 64 rows for latent dimensions
//             128dq..128dq+127 (each V^T tile read from LDS once, used for both
//             32-row tiles); they own the output accumulator, copy the pages
//             into LDS and write the piece results.
// One workgroup barrier opens each period k.  In period k the QK waves turn
// block k into probability codes and per-row state, publish them in LDS and
// raise their flags; the PV waves meanwhile run the products of block k-1 (their
// operands already in registers), issue the copies, take block k's V^T tiles
// into registers, wait for the QK flags and take block k's codes and state.  So
// the products of a block run at the top of the next period, the latent stage of
// block k-1 is free when period k opens, and the code/state buffers are single
// (the PV waves have read them before the barrier after which the QK waves write
// them again).  (The paper's Hopper kernel splits the work between two warp
// groups, Algorithm 1 and Appendix E; here the split is by phase instead of by
// output half.)
//
// Data movement: each 64-token page (32 KiB E4M3 latent, 8 KiB bf16 RoPE,
// 256 B scales) is copied HBM -> LDS with 16-byte direct-to-LDS loads, issued
// once per period by the PV waves (after the products of block k-1 with one row
// group, right after the barrier with several): the latent three blocks ahead of
// the QK waves, the RoPE/scale part two.  The latent lives four periods in LDS
// (three arriving, one in use) and the RoPE/scale part three, hence a 4-stage
// latent ring and a 3-stage RoPE/scale ring (158 KiB of LDS in all).  Latent rows are
// stored with the 16-byte chunk index XOR-swizzled by the token index (swz) so
// that both the token-major QK reads and the transposed PV reads avoid bank
// conflicts.  Page ids travel the same way, requested three periods before the
// latent copy that uses them.  A workgroup starts from the descriptor of its block
// range that the prep kernel wrote (range and first sequence): no search of the
// split plan.  When the range crosses into another sequence, the QK waves fetch
// its bounds two blocks ahead and load its queries right after publishing the
// previous sequence's last block.
// Two PV-wave schedules (template flag kRotate, chosen by the launch): with one
// row group, products of block k-1 first, then the copies, then the transposed
// reads of block k into the same registers; with several row groups (pages shared
// through L2, the period bound by the waves' own work), copies first, products,
// then the transposed reads into a rotating set of six register slots, so that no
// read waits for a product still reading its destination.
//
// Per block (matrices transposed so that one lane owns one query row):
//   S^T[16 tok x 16 rows]  = K_c^T . q8^T   (16x16x128 FP8 MFMA, K = 512), 4 token tiles
//                          + K_r^T . q_r^T  (16x16x32 BF16 MFMA, K = 64)
//   s = log2(e) tau (sigma_q sigma_K acc_c + acc_r)   (Section 3.1 domain alignment,
//       applied to the two accumulators instead of pre-scaling the RoPE operands)
//   running max m, block scale sigma_P = max(max(e sigma_K) / 448, 2^-40),
//   gamma = exp(m_old - m) sigma_p_old / sigma_P, l = gamma l + sum(e) / sigma_P,
//   codes pi = E4M3(e sigma_K / sigma_P)                 (Appendix D)
//   O^T[128 dims x 64 rows] = gamma O^T + V^T . P^T       (FP8 MFMA, K = 64 tokens)
// V^T is read straight from the token-major latent tile with the LDS transpose
// read (ds_read_b64_tr_b8; the CDNA counterpart of the paper's V-tile
// transposition).  The K (token) order of the PV product is chosen so that each
// QK lane's 16 codes are one contiguous 16-byte piece of a PV lane's B operand,
// and the transposed reads fetch V rows in that same order: no accumulator
// permutation is needed.  Blocks are consumed in increasing order,
// the monotone order of Appendix E.  Slots past the end of a sequence hold
// stale bytes; their logits are masked to -inf, their fused probabilities
// forced to 0 and their V bytes cleared before the PV product.

#include "piece_end.h"
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
constexpr int kXcBytes = 64 * 64;               // probability codes [row][64 token slots]; 16-byte
                                                // chunk c of row r at chunk c ^ ((r >> 2) & 3), so that
                                                // 16 consecutive rows hit 16 distinct bank groups
constexpr int kXgBytes = 2 * 32 * 16;           // per-row gamma, l, m, sigma_p [rt][row] x float4
constexpr int kXfBytes = 4 * 4;                 // handshake flags of the QK waves
constexpr int kXpBytes = 4 * 4 * 4;             // page-id ring of the PV waves [wave][4 slots]
constexpr int kXpBase = kXBase + kXcBytes + kXgBytes + kXfBytes;
constexpr int kSmemBytes = kXpBase + kXpBytes;
static_assert(kSmemBytes <= 160 * 1024, "LDS budget of one workgroup");
constexpr float kLn2 = 0.69314718055994531f;
static_assert(20 + kPieceStores < 64, "wait counter range");

// Branch weights for the block layout: the rare cases of a period (a piece start
// or end, a sequence's last page, the first and last periods) are laid out off the
// straight path, which then runs with fewer taken branches.
// (macros: the hint must sit in the branch condition itself to reach the layout)
#define likely(c) __builtin_expect(!!(c), 1)
#define unlikely(c) __builtin_expect(!!(c), 0)

// Latent rows are stored with 16-byte chunk c of token t at chunk c ^ swz(t),
// RoPE rows with chunk c at c ^ rswz(t).  Sixteen consecutive tokens (the QK
// operand reads) map a given chunk to sixteen distinct 16-byte bank groups, and
// the eight tokens of one transposed-read group (PV reads: t0..t0+3 and
// t0+16..t0+19) to eight distinct groups of a 128-byte line.
__device__ __forceinline__ int swz(int t) { return (t & 15) ^ (((t >> 4) & 1) << 2); }
__device__ __forceinline__ int rswz(int t) { return (t >> 1) & 7; }

// Per-row results at a piece end from the published state {gamma, l, m, sigma_P} of
// the row's last block: 1/l and LSE = ln 2 (m + log2(sigma_P l)) (m in log2 units;
// Algorithm 1 finalisation); 0 and -inf for a row without tokens, NaN for a bad piece.
__device__ __forceinline__ void piece_row_results(v4f gl0, v4f gl1, bool bad, float (&inv)[2], float (&lse)[2]) {
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const v4f gl = r == 0 ? gl0 : gl1;
    const float lfin = gl[1];
    const bool empty = !(lfin > 0.0f);
    inv[r] = empty ? 0.0f : 1.0f / lfin;
    lse[r] = empty ? -INFINITY : (gl[2] + log2f(gl[3] * lfin)) * kLn2;
    if (bad) {
      inv[r] = __builtin_nanf("");
      lse[r] = __builtin_nanf("");
    }
  }
}

// Handshake flags in LDS.  A wave's LDS operations complete in issue order, so
// a flag stored after lds_wait_all() is seen only after the data stored before it.
// (the builtin rather than inline asm: the compiler's own wait-count pass then
// knows that every LDS result is in, and inserts no later waits for them)
__device__ __forceinline__ void lds_wait_all() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);            // lgkmcnt(0); vmcnt and expcnt left alone
  asm volatile("" ::: "memory");
}
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
// all four QK waves have published block k
__device__ __forceinline__ bool flags_past(v4i f4, int k) { return f4[0] > k && f4[1] > k && f4[2] > k && f4[3] > k; }

template <bool kRotate, bool kExact>
__global__ __launch_bounds__(512, 1) void decode_kernel(DecodeArgs a, const int32_t* __restrict__ prefix,
                                                        const int32_t* __restrict__ page_table,
                                                        const int32_t* __restrict__ seq_lens) {
  __shared__ __attribute__((aligned(1024))) uint8_t smem[kSmemBytes];
  uint8_t* xc = smem + kXBase;                                                 // [64 rows][64] codes
  float* xg = reinterpret_cast<float*>(smem + kXBase + kXcBytes);               // [64 rows] x 4
  int* xf = reinterpret_cast<int*>(smem + kXBase + kXcBytes + kXgBytes);        // QK flags

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

  // ---- the global block range of this workgroup and its first piece, from the
  // start descriptor the prep kernel wrote (one scalar load, no search) ------
  const int32_t* dsc = a.desc + (int64_t)unit * kDescInts;
  const int gstart = dsc[kDescStart], gend = dsc[kDescEnd];
  if (gstart >= gend) return;
  const int nblocks = gend - gstart;

  // piece bookkeeping (identical in every wave; scalar): the piece of the current
  // block, and the next one, fetched a period before it starts
  int cur_b = dsc[kDescSeq], cur_p0 = dsc[kDescP0], cur_end = dsc[kDescP1], cur_n = dsc[kDescLen];
  int cur_blk0 = gstart - cur_p0;
  int nx_b = 0, nx_p0 = 0, nx_end = 0, nx_n = 0;
  // (the three loads of the usual case, the next sequence, are issued together:
  // one memory round trip per piece; only sequences without blocks loop)
  auto fetch_next = [&](int gb) {                 // gb: first block of the next piece
    int b = cur_b + 1;
    int p0 = prefix[b], p1 = prefix[b + 1], nb = seq_lens[b];
    asm volatile("" ::"s"(nb));                   // keeps the length load beside the prefix loads
    while (p1 <= gb) {
      ++b;
      p0 = p1;
      p1 = prefix[b + 1];
      nb = seq_lens[b];
    }
    nx_b = b;
    nx_p0 = p0;
    nx_end = p1;
    nx_n = nb;
  };
  auto take_next = [&](int gb) {
    cur_b = nx_b;
    cur_p0 = nx_p0;
    cur_blk0 = gb - nx_p0;
    cur_end = nx_end;
    cur_n = nx_n;
  };

  if (is_qk && lane == 0) flag_store(xf + w, 0);   // ordered before any wait by the first barrier

  if (is_qk) {
    // ======================= QK / softmax waves ==============================
    // lane (n16, g4): row 16w + n16; its 16 logits per block are the tokens
    // 16t + 4g4 + v of the four 16-token tiles t (v = 0..3)
    const int n16 = lane & 15, g4 = lane >> 4;
    const int row = 64 * g + 16 * w + n16;         // query row of this lane within the sequence
    const bool row_ok = row < a.R;
    const float sl2 = a.sl2;
    float cq = 0.f;                 // sigma_q
    // q8 bytes 128s + 32g4 .. +31: qv[s] is the B operand of FP8 K-step s; with exact
    // accumulation qh[4s + j] holds bytes 128s + 32g4 + 8j .. +7 as halfs, the B
    // operand of F16 step 4s + j
    v8i qv[4];
    v4i qh[kExact ? 16 : 1];
    v4i qr[2];                      // q_rope elements 32s + 8g4 .. +7
    float m = -INFINITY, sp = 1.0f, l = 0.0f;
    int vis = 0;
    // per-lane LDS byte offsets inside a stage (constant across blocks):
    //   latent chunk of K-step s, half c of token tile t:
    //     8192 t + (koff[t & 1][c] ^ 128 s)       (swz folded in)
    //   RoPE chunk of step s of tile t:  2048 t + roff[s];  scales: 64 t + soff
    uint32_t koff[2][2], roff[2];
#pragma unroll
    for (int par = 0; par < 2; ++par) {
#pragma unroll
      for (int c = 0; c < 2; ++c)
        koff[par][c] = (uint32_t)((n16 * kDc + (((2 * g4 + c) ^ (n16 & 7) ^ (4 * par)) << 4)) | (128 * (n16 >> 3)));
    }
#pragma unroll
    for (int s = 0; s < 2; ++s) roff[s] = (uint32_t)(n16 * (kDr * 2) + (((4 * s + g4) ^ (n16 >> 1)) << 4));
    const uint32_t soff = (uint32_t)(kRopeBytes + 16 * g4);

    // queries of a piece: for the first piece before the first barrier; for a later
    // one right after the previous piece's last block was published (its queries are
    // no longer read), so the loads overlap the wait at the barrier.  The later
    // piece's bounds are fetched two blocks ahead, after a publication as well, so
    // the scalar round trip is not on the query loads' path.
    auto load_q = [&](int qb) {
      if (row_ok) {
        const int64_t qrow = (int64_t)qb * a.R + row;
        const v4i* src = reinterpret_cast<const v4i*>(a.q8 + qrow * kDc);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const v4i lo4 = src[8 * s + 2 * g4], hi4 = src[8 * s + 2 * g4 + 1];
          if constexpr (kExact) {
            qh[4 * s + 0] = e4m3x8_to_f16(lo4[0], lo4[1]);
            qh[4 * s + 1] = e4m3x8_to_f16(lo4[2], lo4[3]);
            qh[4 * s + 2] = e4m3x8_to_f16(hi4[0], hi4[1]);
            qh[4 * s + 3] = e4m3x8_to_f16(hi4[2], hi4[3]);
          } else {
            qv[s] = v8i{lo4[0], lo4[1], lo4[2], lo4[3], hi4[0], hi4[1], hi4[2], hi4[3]};
          }
        }
        const v4i* rsrc = reinterpret_cast<const v4i*>(a.q_rope + qrow * kDr);
#pragma unroll
        for (int s = 0; s < 2; ++s) qr[s] = rsrc[4 * s + g4];
        cq = a.sq[qrow];
      } else {
#pragma unroll
        for (int s = 0; s < 4; ++s) qv[s] = v8i{0, 0, 0, 0, 0, 0, 0, 0};
        if constexpr (kExact) {
#pragma unroll
          for (int s = 0; s < 16; ++s) qh[s] = v4i{0, 0, 0, 0};
        }
#pragma unroll
        for (int s = 0; s < 2; ++s) qr[s] = v4i{0, 0, 0, 0};
        cq = 0.f;
      }
    };
    auto reset_rows = [&]() {
      vis = a.causal ? cur_n - a.q_len + 1 + row / a.H : cur_n;
      m = -INFINITY; sp = 1.0f; l = 0.0f;
    };
    load_q(cur_b);
    reset_rows();
    bool nx_ready = false, q_ready = false;   // next piece's bounds fetched / its queries loaded

    for (int k = 0; k < nblocks; ++k) {
      barrier_vm_lgkm0<63>();                              // page k has landed (PV waves waited)
      const int gb = gstart + k;
      if (unlikely(gb >= cur_end)) {                                 // first block of a later piece
        if (!q_ready) {
          if (!nx_ready) fetch_next(gb);
          load_q(nx_b);
        }
        take_next(gb);
        reset_rows();
        nx_ready = q_ready = false;
      }
      const int blk = gb - cur_p0;
      const uint8_t* st = smem + (k % kLatStages) * kLatBytes;             // latent of block k
      const uint8_t* sr = smem + kRsBase + (k % kRsStages) * kRsBytes;     // its RoPE and scales

      // ---- S^T tiles = K . Q^T, token tile by token tile; the operands of tiles
      // t+1 (and t+2) are requested before the products of tile t
      v4f skq[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) skq[t] = *reinterpret_cast<const v4f*>(sr + soff + 64 * t);
      v4f accC[4], accR[4];
      v4i kc[2][4][2], kr[2][2];
      auto load_tile = [&](int t, int slot) {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
#pragma unroll
          for (int c = 0; c < 2; ++c)
            kc[slot][s][c] = *reinterpret_cast<const v4i*>(st + 8192 * t + (koff[t & 1][c] ^ (uint32_t)(128 * s)));
        }
#pragma unroll
        for (int s = 0; s < 2; ++s) kr[slot][s] = *reinterpret_cast<const v4i*>(sr + 2048 * t + roff[s]);
      };
      load_tile(0, 0);
      load_tile(1, 1);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int slot = t & 1;
        v4f c4 = v4f{0.f, 0.f, 0.f, 0.f}, r4 = v4f{0.f, 0.f, 0.f, 0.f};
        if constexpr (kExact) {
          // exact accumulation: each lane's 32 codes of a 128-dim step feed four
          // 16x16x32 F16 MFMAs (codes converted exactly, the q operand in the same
          // dimension order), accumulated in float32
#pragma unroll
          for (int s = 0; s < 4; ++s) {
            c4 = mfma_f16_16x16x32(e4m3x8_to_f16(kc[slot][s][0][0], kc[slot][s][0][1]), qh[4 * s + 0], c4);
            c4 = mfma_f16_16x16x32(e4m3x8_to_f16(kc[slot][s][0][2], kc[slot][s][0][3]), qh[4 * s + 1], c4);
            c4 = mfma_f16_16x16x32(e4m3x8_to_f16(kc[slot][s][1][0], kc[slot][s][1][1]), qh[4 * s + 2], c4);
            c4 = mfma_f16_16x16x32(e4m3x8_to_f16(kc[slot][s][1][2], kc[slot][s][1][3]), qh[4 * s + 3], c4);
          }
        } else {
          // FP8 MFMA: the hardware sums each group of eight consecutive K positions
          // with every product truncated to a multiple of 2^(E-13), E the group's
          // largest exponent sum (the accuracy the parity tests allow for this mode)
#pragma unroll
          for (int s = 0; s < 4; ++s)
            c4 = mfma_f8_16x16x128(v8i{kc[slot][s][0][0], kc[slot][s][0][1], kc[slot][s][0][2], kc[slot][s][0][3],
                                       kc[slot][s][1][0], kc[slot][s][1][1], kc[slot][s][1][2], kc[slot][s][1][3]},
                                   qv[s], c4);
        }
#pragma unroll
        for (int s = 0; s < 2; ++s) r4 = mfma_bf16_16x16x32(kr[slot][s], qr[s], r4);
        accC[t] = c4;
        accR[t] = r4;
        if (t + 2 < 4) load_tile(t + 2, slot);
        __builtin_amdgcn_sched_barrier(0);
      }

      // ---- block statistics of this row (16 logits here, 48 in lanes n16 + 16 g')
      float sk[16], pp[16];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          sk[4 * t + v] = skq[t][v];
          // raw logit u = sigma_q sigma_K acc_c + acc_r; s = tau log2(e) u enters the
          // exponentials through one fma each
          pp[4 * t + v] = fmaf(accC[t][v], cq * skq[t][v], accR[t][v]);
        }
      }
      const bool tail = (blk + 1) * kPage > vis;   // some token of this block is hidden from this row
      if (unlikely(tail)) {
        // hidden tokens and stale slots past the sequence end: logit -inf, scale 0
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int j = blk * kPage + 16 * (i >> 2) + 4 * g4 + (i & 3);
          const bool vis_j = j < vis;
          pp[i] = vis_j ? pp[i] : -INFINITY;
          sk[i] = vis_j ? sk[i] : 0.0f;
        }
      }
      // (maxima that propagate NaN: no logit is NaN here -- hidden and stale slots are -inf,
      // and a bad page marks the piece NaN whatever its logits)
      const float mb = quad_vmax(vmax16(pp)) * sl2;  // block max of this row (log2 units)
      v4i mine = v4i{0, 0, 0, 0};
      float gam = 1.0f;
      if (likely(mb > -INFINITY)) {                        // the row sees a token of this block
        const float m_new = vmax(m, mb);
        float e[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) e[i] = __builtin_amdgcn_exp2f(fmaf(pp[i], sl2, -m_new));
#pragma unroll
        for (int i = 0; i < 16; ++i) pp[i] = e[i] * sk[i];
        float esum = ((e[0] + e[1]) + (e[2] + e[3])) + ((e[4] + e[5]) + (e[6] + e[7]));
        esum += ((e[8] + e[9]) + (e[10] + e[11])) + ((e[12] + e[13]) + (e[14] + e[15]));
        float pmax = vmax16(pp);
        esum = quad_sum(esum);
        pmax = quad_vmax(pmax);
        // (reciprocals instead of divisions: off by at most an ulp, far inside the
        // rounding slack of the probability codes)
        const float sP = fmaxf(pmax * (1.0f / kFp8Max), kEps);
        const float inv = __builtin_amdgcn_rcpf(sP);
        gam = __builtin_amdgcn_exp2f(m - m_new) * (sp * inv);
        l = gam * l + esum * inv;
        m = m_new;
        sp = sP;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          int wd = cvt_pk_e4m3(pp[4 * t + 0] * inv, pp[4 * t + 1] * inv, 0, false);
          wd = cvt_pk_e4m3(pp[4 * t + 2] * inv, pp[4 * t + 3] * inv, wd, true);
          mine[t] = wd;
        }
      }
      // codes of tokens 16t + 4g4 + v at byte 16 g4 + 4t + v of the row (logical; the
      // 16-byte chunk g4 sits at chunk g4 ^ ((row >> 2) & 3)); the PV
      // waves read the previous block's before this period's barrier
      *reinterpret_cast<v4i*>(xc + (16 * w + n16) * 64 + 16 * (g4 ^ ((n16 >> 2) & 3))) = mine;
      if (g4 == 0) *reinterpret_cast<v4f*>(xg + (16 * w + n16) * 4) = v4f{gam, l, m, sp};
      lds_wait_all();
      if (lane == 0) flag_store(xf + w, k + 1);   // block k published
      if (unlikely(cur_end < gend)) {                        // a later piece starts inside the range
        if (!nx_ready && gb + 2 >= cur_end) {
          fetch_next(cur_end);
          nx_ready = true;
        }
        if (gb + 1 == cur_end) {                   // this piece's queries are no longer read
          load_q(nx_b);
          q_ready = true;
        }
      }
    }
    barrier_vm_lgkm0<63>();                        // pairs with the PV waves' last top barrier
  } else {
    // =========================== PV waves ====================================
    const int dq = __builtin_amdgcn_readfirstlane(w - 4);   // dims 128dq..128dq+127; wave-uniform
    const int row0 = 64 * g + n, row1 = row0 + 32;          // query rows of this lane (row tiles 0, 1)
    // This wave copies latent rows 16dq..16dq+15 (instruction j: rows 16dq + 2j + h,
    // LDS chunk n of the row takes global chunk n ^ swz(row)), RoPE rows
    // 16dq..16dq+15 and scales 16dq..16dq+15 of each page.  For row t = 16dq + 2j + h,
    // n ^ swz(t) = (n ^ h) ^ cj with the wave-uniform cj = 2j ^ 4(dq & 1), so one
    // per-lane register serves all eight latent copies:
    //   global offset = (16dq + 2j) * 512 + (lat_v ^ (cj << 4)).
    const uint32_t lat_v = (uint32_t)((((n ^ h) << 4)) | (h << 9));
    // RoPE instruction j covers rows 16dq + 8j + lane/8; LDS chunk lane%8 takes global
    // chunk (lane%8) ^ rswz(row) = (lane%8) ^ ((lane/16) & 3) ^ 4j:
    //   global offset = (16dq + 8j) * 128 + (rope_v ^ (j << 6)).
    const uint32_t rope_v = (uint32_t)((lane >> 3) * (kDr * 2) + (((lane & 7) ^ ((lane >> 4) & 3)) << 4));
    const uint32_t sc_off = (uint32_t)((16 * dq + (lane & 15)) * 4);
    const uint32_t smem_base = lds_offset(smem);

    // page-table cursor (scalar): the next block asked for lies in sequence ib,
    // whose blocks are global blocks [ib_lo, ib_hi).  Blocks are asked for in
    // nondecreasing order; past the range the last block stands in.
    int ib = cur_b, ib_lo = cur_p0, ib_hi = cur_end;
    auto page_entry = [&](int kb) -> const int32_t* {
      const int gb = gstart + min(kb, nblocks - 1);
      while (unlikely(gb >= ib_hi)) {                        // skips sequences without blocks
        ++ib;
        ib_lo = ib_hi;
        ib_hi = prefix[ib + 1];
      }
      return page_table + (int64_t)ib * a.max_pages + (gb - ib_lo);
    };
    // In the loop, page ids come through the copy path rather than the scalar
    // cache: a scalar load shares its wait counter with the LDS reads, so every
    // LDS wait of the period would also wait for it, a full memory round trip
    // under the copy traffic.  In each copying period k every PV wave requests
    // (one lane, one dword) the id of block k+6 into slot (k+6) % 4 of its ring;
    // the request is complete at the top of period k+2, at whose end the slot is
    // read (the id of the latent copy of period k+3).  A slot is read before it
    // is requested again.
    const uint32_t pg_ring = smem_base + kXpBase + 16 * dq;
    const int* pg_ring_p = reinterpret_cast<const int*>(smem + kXpBase + 16 * dq);
    auto request_page = [&](int kb) {
      const int32_t* e = page_entry(kb);            // cursor update in uniform control flow
      if (lane == 0) g2lds4_so(reinterpret_cast<const uint8_t*>(e), 0u, pg_ring + 4 * (kb & 3));
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
        const uint32_t cj = (uint32_t)(((2 * i) ^ (4 * (dq & 1))) << 4);
        g2lds16_so(src + (16 * dq + 2 * i) * kDc, lat_v ^ cj, dst + 1024 * (8 * dq + i));
      }
    };
    auto copy_rope_scale = [&](int kb, int page) {
      if (!page_ok(page)) page = 0;
      const uint8_t* rp = reinterpret_cast<const uint8_t*>(a.k_rope) + (int64_t)page * kRopeBytes;
      const uint8_t* sc = reinterpret_cast<const uint8_t*>(a.kv_scale) + (int64_t)page * kScBytes;
      const uint32_t dst = smem_base + kRsBase + (kb % kRsStages) * kRsBytes;
#pragma unroll
      for (int i = 0; i < 2; ++i)
        g2lds16_so(rp + (16 * dq + 8 * i) * (kDr * 2), rope_v ^ (uint32_t)(i << 6), dst + 1024 * (2 * dq + i));
      if (lane < 16) g2lds4_so(sc, sc_off, dst + kRopeBytes + 64 * dq);
    };
    // Copy requests, in issue order.  Prologue: page ids 4 and 5, latent+RoPE of
    // blocks 0 and 1, latent of block 2.  Period k (while k + 2 < nblocks): page
    // id k+6, RoPE of block k+2, latent of block k+3: 1 + 3 + 8 = 12 requests.
    // Requests for blocks past the range repeat the last block's page into the
    // stage that block would take, which nothing reads afterwards.
    // (the cursor only moves forward: blocks are asked for in increasing order)
    int pg_rope, pg_lat;                           // ids of the RoPE and latent copies of the period
    {
      const int pg0 = *page_entry(0);
      const int pg1 = *page_entry(1);
      pg_rope = *page_entry(2);
      pg_lat = *page_entry(3);
      request_page(4);
      request_page(5);
      copy_latent(0, pg0);
      copy_rope_scale(0, pg0);
      copy_latent(1, pg1);
      copy_rope_scale(1, pg1);
      copy_latent(2, pg_rope);
    }

    // O[2T + r]: O^T tile of dims 128dq + 32T.. and row tile r
    v16f O[8];
#pragma unroll
    for (int T = 0; T < 8; ++T) O[T] = v16f{0};

    // transposed V reads: 16-lane group g16 of half h reads 8 token rows x 16 bytes;
    // lane pair (2i, 2i+1) supplies row i.  K index 32h + 8c + i of the PV product
    // is token 32(c&1) + 16(i>>2) + 8h + 4(c>>1) + (i&3): the token whose code the
    // QK waves store at byte 32h + 8c + i of the row.  The byte offset of tile T,
    // read c inside a stage is tr_off[c] ^ (T << 5): the row offset, byte half and
    // swizzled chunk ((8dq + g16) ^ swz(tok)) ^ 2T occupy disjoint bits, and so
    // does the stage base.
    const int q16 = lane & 15, tri = q16 >> 1, trb = q16 & 1, g16 = (lane >> 4) & 1;
    uint32_t tr_off[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int tok = 32 * (c & 1) + 16 * (tri >> 2) + 8 * h + 4 * (c >> 1) + (tri & 3);
      tr_off[c] = (uint32_t)(tok * kDc + 8 * trb) | (uint32_t)(((8 * dq + g16) ^ swz(tok)) << 4);
    }
    if constexpr (!kRotate) {
      // Top-of-period wait: block k (latent and RoPE) complete, and the page id
      // read at the end of the period.  Loads complete in issue order: in steady
      // state the RoPE copy of block k is followed by the latent copy of block k+1,
      // the piece-end stores of period k-1 if any (kPieceStores of them) and its 12
      // requests, so "at most 20 (+ kPieceStores) outstanding" suffices; 19 in
      // period 0, after the prologue.
      auto top_barrier = [&](int k, bool after_stores) {
        if (unlikely(k + 1 >= nblocks)) barrier_vm_lgkm0<0>();
        else if (unlikely(k == 0)) barrier_vm_lgkm0<19>();
        else if (unlikely(after_stores)) barrier_vm_lgkm0<20 + kPieceStores>();
        else barrier_vm_lgkm0<20>();
      };

      v2i rv[4][4];                 // V^T tiles of the pending block
      v8i P0, P1;                   // its codes, row tiles 0 and 1
      v4f gl0, gl1;                 // its per-row state {gamma, l, m, sigma_P}
      bool cur_bad = false;
      bool stored = false;          // the previous period wrote piece results
      for (int k = 0;; ++k) {
        top_barrier(k, stored);
        stored = false;
        if (likely(k > 0)) {
          // ---- PV of block k-1 --------------------------------------------------
          // each accumulator is rescaled right before its product, so that the
          // multiplies of the next one run while the matrix core works
  #pragma unroll
          for (int T = 0; T < 4; ++T) {
            const v8i A = v8i{rv[T][0][0], rv[T][0][1], rv[T][1][0], rv[T][1][1],
                              rv[T][2][0], rv[T][2][1], rv[T][3][0], rv[T][3][1]};
            O[2 * T] *= gl0[0];
            O[2 * T] = mfma_f8_32x32x64(A, P0, O[2 * T]);
            __builtin_amdgcn_sched_barrier(0);
            O[2 * T + 1] *= gl1[0];
            O[2 * T + 1] = mfma_f8_32x32x64(A, P1, O[2 * T + 1]);
            __builtin_amdgcn_sched_barrier(0);
          }
          // ---- end of a piece: write the normalized partial output and LSE ----
          // (one 16-byte store at a time; a bad page id makes the multiplier NaN)
          if (unlikely(k == nblocks || gstart + k >= cur_end)) {
            // the piece of block k-1 ends: exactly kPieceStores stores (the next
            // top-of-period wait counts them); every wave writes the same LSEs
            const int64_t pid = a.chunk_blocks == 0 ? (int64_t)unit + cur_b
                                                    : (int64_t)cur_b * a.num_splits + cur_blk0 / a.chunk_blocks;
            const bool whole = cur_blk0 == 0 && gstart + k >= cur_end;   // the piece is its whole sequence
            float inv[2], lse[2];
            piece_row_results(gl0, gl1, cur_bad, inv, lse);
            store_piece(a, O, inv[0], inv[1], lse[0], lse[1], row0, row1, dq, h, pid, cur_b, whole);
  #pragma unroll
            for (int T = 0; T < 8; ++T) O[T] = v16f{0};
            stored = true;
          }
        }
        // copies after the products and the piece-end stores, so that the stores
        // precede the period's copies in the wait counter
        if (likely(k + 2 < nblocks)) {
          request_page(k + 6);
          copy_rope_scale(k + 2, pg_rope);
          copy_latent(k + 3, pg_lat);
          pg_rope = pg_lat;
        }
        if (unlikely(k == nblocks)) break;

        // ---- block k: piece bookkeeping (mirrors the QK waves) -----------------
        const int gb = gstart + k;
        if (unlikely(gb >= cur_end)) {
          fetch_next(gb);
          take_next(gb);
          cur_bad = false;
        }
        cur_bad |= ((stage_bad >> (k % kLatStages)) & 1u) != 0;
        const int valid = min(kPage, cur_n - (gb - cur_p0) * kPage);
        uint8_t* stp = smem + (k % kLatStages) * kLatBytes;
        if (unlikely(valid < kPage)) {
          // last page of a sequence: clear the bytes of the slots past its end that
          // this wave reads (stale data could hold NaN codes; their probability
          // codes are 0).  The QK waves mask these slots whatever they hold.
          const int nz = (kPage - valid) * 8;
          for (int i = lane; i < nz; i += 64) {
            const int t = valid + (i >> 3);
            const int c = 8 * dq + (i & 7);
            *reinterpret_cast<v4i*>(stp + t * kDc + ((c ^ swz(t)) << 4)) = v4i{0, 0, 0, 0};
          }
        }
        // V^T tiles of block k
        const uint32_t st_lds = smem_base + (k % kLatStages) * kLatBytes;
  #pragma unroll
        for (int T = 0; T < 4; ++T) {
  #pragma unroll
          for (int c = 0; c < 4; ++c) rv[T][c] = lds_read_tr8_at((st_lds | tr_off[c]) ^ (uint32_t)(T << 5));
        }
        // codes and state of block k, once all four QK waves have published them
        {
          // one exit for both ends of the wait (the flags seen, or the bound reached),
          // decided again from the last poll: codes never published, or a zero
          // bound, mark the piece, which then comes out NaN
          v4i f4;
          int spin = 0;
          do {
            f4 = flag_load4(xf);
          } while (!flags_past(f4, k) && ++spin < a.spin_limit);
          if (!flags_past(f4, k) || a.spin_limit <= 0) cur_bad = true;
        }
        asm volatile("" ::: "memory");
        gl0 = *reinterpret_cast<const v4f*>(xg + n * 4);
        gl1 = *reinterpret_cast<const v4f*>(xg + (n + 32) * 4);
        // B operand of row tile r: bytes 32h .. 32h+31 of row 32r + n (the K order
        // of the PV product, see the transposed reads)
        const int cs = (n >> 2) & 3;                  // chunk swizzle of rows n and 32 + n
        const v4i c00 = *reinterpret_cast<const v4i*>(xc + n * 64 + 16 * ((2 * h) ^ cs));
        const v4i c01 = *reinterpret_cast<const v4i*>(xc + n * 64 + 16 * ((2 * h + 1) ^ cs));
        const v4i c10 = *reinterpret_cast<const v4i*>(xc + (32 + n) * 64 + 16 * ((2 * h) ^ cs));
        const v4i c11 = *reinterpret_cast<const v4i*>(xc + (32 + n) * 64 + 16 * ((2 * h + 1) ^ cs));
        P0 = v8i{c00[0], c00[1], c00[2], c00[3], c01[0], c01[1], c01[2], c01[3]};
        P1 = v8i{c10[0], c10[1], c10[2], c10[3], c11[0], c11[1], c11[2], c11[3]};
        const int pg_next = pg_ring_p[(k + 4) & 3];   // id of block k+4 (stale when not copied)
        lds_wait_all();
        pg_lat = __builtin_amdgcn_readfirstlane(pg_next);
      }
    } else {
      // Top-of-period wait: block k (latent and RoPE) complete, and the page id
      // read at the end of the period.  Loads complete in issue order.  Each period
      // issues its 12 requests first and the piece-end stores, if any, after them, so
      // in steady state the RoPE copy of block k (period k-2) is followed by the
      // latent copy of block k+1, the stores of period k-2, the 12 requests of period
      // k-1 and its stores: "at most 20 (+ kPieceStores per storing period)
      // outstanding" suffices (capped at the counter's range, which only waits
      // longer); 19 in period 0, after the prologue.
      auto top_barrier = [&](int k, int storing_periods) {
        if (unlikely(k + 1 >= nblocks)) barrier_vm_lgkm0<0>();
        else if (unlikely(k == 0)) barrier_vm_lgkm0<19>();
        else if (likely(storing_periods == 0)) barrier_vm_lgkm0<20>();
        else if (storing_periods == 1) barrier_vm_lgkm0<20 + kPieceStores>();
        else barrier_vm_lgkm0<63>();
      };

      // V^T tiles in six 8-register slots: tile T of block k-1 sits in old[T]; the
      // transposed reads of block k, issued after the products of block k-1, go to
      // two free slots (tiles 0, 1) and to the slots of tiles 0 and 1 of block k-1
      // (tiles 2, 3).  So no read waits for a product still reading its destination,
      // and the slot roles rotate with period 3.
      v2i sA[4], sB[4], sC[4], sD[4], sE[4], sF[4];
      v8i P0, P1;                   // codes of the pending block, row tiles 0 and 1
      v4f gl0, gl1;                 // its per-row state {gamma, l, m, sigma_P}
      bool cur_bad = false;
      bool st1 = false, st2 = false;   // periods k-1 and k-2 wrote piece results
      auto period = [&](int k, v2i (&o0)[4], v2i (&o1)[4], v2i (&o2)[4], v2i (&o3)[4], v2i (&f0)[4],
                        v2i (&f1)[4]) -> bool {
        const bool PV = k > 0, RD = k < nblocks;   // products of block k-1, reads of block k
        top_barrier(k, (st1 ? 1 : 0) + (st2 ? 1 : 0));
        st2 = st1;
        st1 = false;
        if (likely(k + 2 < nblocks)) {
          request_page(k + 6);
          copy_rope_scale(k + 2, pg_rope);
          copy_latent(k + 3, pg_lat);
          pg_rope = pg_lat;
        }
        // the piece that block k-1 closes, if any (before the bookkeeping of block k)
        const bool close = PV && (!RD || gstart + k >= cur_end);
        const int64_t pid = a.chunk_blocks == 0 ? (int64_t)unit + cur_b
                                                : (int64_t)cur_b * a.num_splits + cur_blk0 / a.chunk_blocks;
        const bool close_bad = cur_bad;
        const int close_b = cur_b;
        if (RD) {
          // ---- block k: piece bookkeeping (mirrors the QK waves) ---------------
          const int gb = gstart + k;
          if (unlikely(gb >= cur_end)) {
            fetch_next(gb);
            take_next(gb);
            cur_bad = false;
          }
          cur_bad |= ((stage_bad >> (k % kLatStages)) & 1u) != 0;
          const int valid = min(kPage, cur_n - (gb - cur_p0) * kPage);
          uint8_t* stp = smem + (k % kLatStages) * kLatBytes;
          if (unlikely(valid < kPage)) {
            // last page of a sequence: clear the bytes of the slots past its end that
            // this wave reads (stale data could hold NaN codes; their probability
            // codes are 0).  The QK waves mask these slots whatever they hold.
            const int nz = (kPage - valid) * 8;
            for (int i = lane; i < nz; i += 64) {
              const int t = valid + (i >> 3);
              const int c = 8 * dq + (i & 7);
              *reinterpret_cast<v4i*>(stp + t * kDc + ((c ^ swz(t)) << 4)) = v4i{0, 0, 0, 0};
            }
          }
        }
        // ---- PV of block k-1, then the V^T reads of block k ---------------------
        const uint32_t st_lds = smem_base + (k % kLatStages) * kLatBytes;
        auto pv_tile = [&](int T, v2i (&src)[4]) {
          const v8i A = v8i{src[0][0], src[0][1], src[1][0], src[1][1], src[2][0], src[2][1], src[3][0], src[3][1]};
          O[2 * T] *= gl0[0];
          O[2 * T] = mfma_f8_32x32x64(A, P0, O[2 * T]);
          __builtin_amdgcn_sched_barrier(0);
          O[2 * T + 1] *= gl1[0];
          O[2 * T + 1] = mfma_f8_32x32x64(A, P1, O[2 * T + 1]);
          __builtin_amdgcn_sched_barrier(0);
        };
        auto tr_tile = [&](int T, v2i (&dst)[4]) {
  #pragma unroll
          for (int c = 0; c < 4; ++c) dst[c] = lds_read_tr8_at((st_lds | tr_off[c]) ^ (uint32_t)(T << 5));
        };
        // all products first, then all reads: tiles 0 and 1 of block k go to the free
        // slots, tiles 2 and 3 to the slots of tiles 0 and 1 of block k-1, whose
        // products are done by the time the later products have been issued
        if (PV) {
          pv_tile(0, o0);
          pv_tile(1, o1);
          pv_tile(2, o2);
          pv_tile(3, o3);
        }
        __builtin_amdgcn_sched_barrier(0);
        if (RD) {
          tr_tile(0, f0);
          tr_tile(1, f1);
          tr_tile(2, o0);
          tr_tile(3, o1);
        }
        __builtin_amdgcn_sched_barrier(0);
        if (PV) {
          // ---- end of a piece: write the normalized partial output and LSE --
          // (one 16-byte store at a time; a bad page id makes the multiplier NaN)
          if (unlikely(close)) {
            // exactly kPieceStores stores (the next top-of-period waits count them)
            float inv[2], lse[2];
            piece_row_results(gl0, gl1, close_bad, inv, lse);
            // (partials only with several row groups: the direct-row stores would raise this
            // schedule's register pressure into spills; the launch leaves out unset)
            store_piece(a, O, inv[0], inv[1], lse[0], lse[1], row0, row1, dq, h, pid, close_b, false);
  #pragma unroll
            for (int T = 0; T < 8; ++T) O[T] = v16f{0};
            st1 = true;
          }
        }
        if (!RD) return false;
        // codes and state of block k, once all four QK waves have published them
        {
          // one exit for both ends of the wait (the flags seen, or the bound reached),
          // decided again from the last poll: codes never published, or a zero
          // bound, mark the piece, which then comes out NaN
          v4i f4;
          int spin = 0;
          do {
            f4 = flag_load4(xf);
          } while (!flags_past(f4, k) && ++spin < a.spin_limit);
          if (!flags_past(f4, k) || a.spin_limit <= 0) cur_bad = true;
        }
        asm volatile("" ::: "memory");
        gl0 = *reinterpret_cast<const v4f*>(xg + n * 4);
        gl1 = *reinterpret_cast<const v4f*>(xg + (n + 32) * 4);
        // B operand of row tile r: bytes 32h .. 32h+31 of row 32r + n (the K order
        // of the PV product, see the transposed reads)
        const int cs = (n >> 2) & 3;                  // chunk swizzle of rows n and 32 + n
        const v4i c00 = *reinterpret_cast<const v4i*>(xc + n * 64 + 16 * ((2 * h) ^ cs));
        const v4i c01 = *reinterpret_cast<const v4i*>(xc + n * 64 + 16 * ((2 * h + 1) ^ cs));
        const v4i c10 = *reinterpret_cast<const v4i*>(xc + (32 + n) * 64 + 16 * ((2 * h) ^ cs));
        const v4i c11 = *reinterpret_cast<const v4i*>(xc + (32 + n) * 64 + 16 * ((2 * h + 1) ^ cs));
        P0 = v8i{c00[0], c00[1], c00[2], c00[3], c01[0], c01[1], c01[2], c01[3]};
        P1 = v8i{c10[0], c10[1], c10[2], c10[3], c11[0], c11[1], c11[2], c11[3]};
        const int pg_next = pg_ring_p[(k + 4) & 3];   // id of block k+4 (stale when not copied)
        lds_wait_all();
        pg_lat = __builtin_amdgcn_readfirstlane(pg_next);
        return true;
      };
      // three periods per iteration: the slot roles rotate without register copies
      for (int k = 0;; k += 3) {
        if (!period(k, sA, sB, sC, sD, sE, sF)) break;        // block k   -> E F A B
        if (!period(k + 1, sE, sF, sA, sB, sC, sD)) break;    // block k+1 -> C D E F
        if (!period(k + 2, sC, sD, sE, sF, sA, sB)) break;    // block k+2 -> A B C D
      }
    }
  }
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream) {
  const int units = a.chunk_blocks == 0 ? a.num_splits : a.B * a.num_splits;
  if (units <= 0) return hipSuccess;
  const int64_t grid = (int64_t)((units + 7) / 8) * 8 * a.G;
  if (grid > 0x7FFFFFFF) return hipErrorInvalidValue;
  // With several row groups the workgroups of a unit share its pages through L2 and
  // the period is bound by the waves' own work: there the copies go first and the
  // products of block k-1 precede the transposed reads of block k (kRotate).  With
  // one row group the pages come from HBM and the products go first.
  auto k = a.G > 1 ? (a.qk_exact ? decode_kernel<true, true> : decode_kernel<true, false>)
                   : (a.qk_exact ? decode_kernel<false, true> : decode_kernel<false, false>);
  hipLaunchKernelGGL(k, dim3((unsigned)grid), dim3(64 * kWaves), 0, stream, a, a.prefix, a.page_table, a.seq_lens);
  return hipGetLastError();
}

}  // namespace snapmla
