// BF16-latent MLA decode: the unquantized baseline of the paper's FP8-vs-BF16
// comparison (Section 4: SnapMLA against a BF16-cache MLA kernel; Section 2,
// absorbed score s = tau (q_nope . c_KV + q_rope . k_rope), V = c_KV).
//
// Cache: kv_latent bf16 [pages][64][512] (1 KiB per token), k_rope bf16
// [pages][64][64]; no scales.  Per 32-token block (one half page):
//   S^T = K . Q^T                  (16x16x32 BF16 MFMA over 576 dims, K = 512 + 64)
//   online softmax: m' = max(m, rowmax s), p = exp(s - m'), l = e^{m-m'} l + sum p
//   O^T = e^{m-m'} O^T + V^T . P^T (32x32x16 BF16 MFMA; P rounded to bf16)
// and per KV piece o = O / l, LSE = m + ln l (natural log of the scaled logits),
// into the same split-KV partials as the FP8 path, merged by snapmla_combine.
//
// Structure as in decode.hip, with 32-token periods so that a latent stage is
// still 32 KiB: 8 waves, QK waves 0-3 (rows 16w..16w+15 against the block's 32
// tokens), PV waves 4-7 (all 64 rows x 128 dims, products of block k-1 at the top
// of period k from operands loaded before the barrier); latent copied three blocks
// ahead into a 4-stage ring, RoPE two blocks ahead into a 3-stage ring, page ids
// through the copy path.  V^T comes from the 16-bit LDS transpose read
// (ds_read_b64_tr_b16: in each 16-lane group, lane 4q + c receives element c of
// the 8-byte pieces addressed by lanes q, q+4, q+8, q+12).

#include "piece_end.h"
#include "snapmla_device.h"
#include "snapmla_internal.h"

namespace snapmla {

namespace {

constexpr int kTok = 32;                        // tokens per block (period)
constexpr int kRowB = 2 * kDc;                  // 1024 B per latent row
constexpr int kLatB = kTok * kRowB;             // 32768
constexpr int kRopeB = kTok * kDr * 2;          // 4096
constexpr int kLatSt = 4;
constexpr int kRopeSt = 3;
constexpr int kRopeBase = kLatSt * kLatB;
constexpr int kPBase = kRopeBase + kRopeSt * kRopeB;    // P bf16 [64 rows][32 tokens]
constexpr int kPBytes = 64 * kTok * 2;
constexpr int kGBase = kPBase + kPBytes;                // per-row {gamma, l, m, 0}
constexpr int kGBytes = 64 * 16;
constexpr int kFBase = kGBase + kGBytes;                // QK flags
constexpr int kRingBase = kFBase + 16;                  // page-id ring [PV wave][4]
constexpr int kSmem = kRingBase + 64;
static_assert(kSmem <= 160 * 1024, "LDS budget of one workgroup");
constexpr int kStores = kPieceStores;                    // piece-end stores of a PV wave
static_assert(18 + kStores < 64, "wait counter range");
constexpr float kLn2f = 0.69314718055994531f;

// Latent rows: 16-byte chunk c of token t at chunk c ^ swz(t).  Within 16
// consecutive tokens swz is a permutation of 0..15 (QK reads: one chunk of 16
// tokens, 16 distinct bank groups); within 4 consecutive tokens from a multiple
// of 4 it keeps bit 0, so a transposed read's 4 tokens x 2 adjacent chunks fall
// in 8 distinct groups.  RoPE rows (128 B): chunk c at c ^ ((t >> 1) & 7).
__device__ __forceinline__ int swz(int t) { return ((t & 3) << 1) | ((t >> 2) & 1) | (t & 8); }

__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
__device__ __forceinline__ void fstore(int* f, int v) {
  __hip_atomic_store(f, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
typedef __attribute__((address_space(3))) volatile v4i lds_v4i_vol;
__device__ __forceinline__ v4i fload4(const int* f) { return *(const lds_v4i_vol*)(f); }

typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;
__device__ __forceinline__ v2i lds_read_tr16_at(uint32_t addr) {
  const v4s r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(uintptr_t)addr);
  return __builtin_bit_cast(v2i, r);
}

__device__ __forceinline__ uint32_t bf16_bits(float x) {
  const uint32_t u = __float_as_uint(x);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__global__ __launch_bounds__(512, 1) void decode_bf16_kernel(DecodeArgs a, const uint16_t* __restrict__ kv_lat,
                                                             const int32_t* __restrict__ prefix,
                                                             const int32_t* __restrict__ page_table,
                                                             const int32_t* __restrict__ seq_lens) {
  __shared__ __attribute__((aligned(1024))) uint8_t smem[kSmem];
  uint8_t* xp = smem + kPBase;
  float* xg = reinterpret_cast<float*>(smem + kGBase);
  int* xf = reinterpret_cast<int*>(smem + kFBase);

  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const bool is_qk = w < 4;
  const int h = lane >> 5, n = lane & 31;

  const int x8 = blockIdx.x & 7, q8i = blockIdx.x >> 3;
  const int g = q8i % a.G;
  const int unit = (q8i / a.G) * 8 + x8;
  const int units = a.chunk_blocks == 0 ? a.num_splits : a.B * a.num_splits;
  if (unit >= units) return;

  // the 64-token block range of this workgroup and its first piece, from the start
  // descriptor the prep kernel wrote (same plan as the FP8 path)
  const int32_t* dsc = a.desc + (int64_t)unit * kDescInts;
  const int gstart = dsc[kDescStart], gend = dsc[kDescEnd];
  if (gstart >= gend) return;
  const int nblk = 2 * (gend - gstart);            // 32-token blocks: two per 64-token block

  int cur_b = dsc[kDescSeq], cur_p0 = dsc[kDescP0], cur_end = dsc[kDescP1], cur_n = dsc[kDescLen];
  int cur_blk0 = gstart - cur_p0;
  auto enter_piece = [&](int gb) {                 // a later piece: sequence cur_b + 1 onwards
    int b = cur_b + 1;
    int p0 = prefix[b], p1 = prefix[b + 1], nb = seq_lens[b];
    asm volatile("" ::"s"(nb));
    while (p1 <= gb) {
      ++b;
      p0 = p1;
      p1 = prefix[b + 1];
      nb = seq_lens[b];
    }
    cur_b = b;
    cur_p0 = p0;
    cur_blk0 = gb - p0;
    cur_end = p1;
    cur_n = nb;
  };

  if (is_qk && lane == 0) fstore(xf + w, 0);

  if (is_qk) {
    // ======================= QK / softmax waves ==============================
    // lane (n16, g4): row 16w + n16; its 8 logits per block are the tokens
    // 16t + 4g4 + v of the two 16-token tiles t (v = 0..3)
    const int n16 = lane & 15, g4 = lane >> 4;
    const int row = 64 * g + 16 * w + n16;
    const bool row_ok = row < a.R;
    const float sl2 = a.sl2;
    v4i qb[18];                     // q bf16 elements 32s + 8g4 .. +7 of K-step s (16 content, 2 RoPE)
    float m = -INFINITY, l = 0.0f;
    int vis = 0;
    // LDS byte offsets inside a stage: latent K-step s of tile t at
    //   ((16t + n16) << 10) | (kx ^ (s << 6)),  kx = 16 ((g4 ^ (sw & 3)) | (sw & 12)), sw = swz(n16)
    // RoPE step s of tile t at 2048 t + roff[s]
    const int sw = swz(n16);
    const uint32_t kx = (uint32_t)(16 * ((g4 ^ (sw & 3)) | (sw & 12)));
    uint32_t roff[2];
#pragma unroll
    for (int s = 0; s < 2; ++s) roff[s] = (uint32_t)(n16 * (kDr * 2) + (((4 * s + g4) ^ (n16 >> 1)) << 4));

    bool fresh = true;                              // the first piece comes from the descriptor
    for (int k = 0; k < nblk; ++k) {
      barrier_vm_lgkm0<63>();
      const int gb = gstart + (k >> 1), hk = k & 1;
      if (fresh || gb >= cur_end) {
        if (!fresh) enter_piece(gb);
        fresh = false;
        vis = a.causal ? cur_n - a.q_len + 1 + row / a.H : cur_n;
        if (row_ok) {
          const int64_t qrow = (int64_t)cur_b * a.R + row;
          const v4i* src = reinterpret_cast<const v4i*>(a.q_nope + qrow * kDc);
#pragma unroll
          for (int s = 0; s < 16; ++s) qb[s] = src[4 * s + g4];
          const v4i* rsrc = reinterpret_cast<const v4i*>(a.q_rope + qrow * kDr);
#pragma unroll
          for (int s = 0; s < 2; ++s) qb[16 + s] = rsrc[4 * s + g4];
        } else {
#pragma unroll
          for (int s = 0; s < 18; ++s) qb[s] = v4i{0, 0, 0, 0};
        }
        m = -INFINITY;
        l = 0.0f;
      }
      const int tok0 = (gb - cur_p0) * kPage + kTok * hk;      // sequence position of the block's token 0
      const uint32_t st = (uint32_t)((k % kLatSt) * kLatB);
      const uint8_t* sr = smem + kRopeBase + (k % kRopeSt) * kRopeB;
      const uint32_t sbase = lds_offset(smem) + st;

      v4f acc[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const uint32_t tb = sbase + (uint32_t)((16 * t + n16) << 10);
        v4i kk[18];
#pragma unroll
        for (int s = 0; s < 16; ++s)
          kk[s] = *(const __attribute__((address_space(3))) v4i*)(uintptr_t)(tb | (kx ^ (uint32_t)(s << 6)));
#pragma unroll
        for (int s = 0; s < 2; ++s) kk[16 + s] = *reinterpret_cast<const v4i*>(sr + 2048 * t + roff[s]);
        v4f c4 = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < 18; ++s) c4 = mfma_bf16_16x16x32(kk[s], qb[s], c4);
        acc[t] = c4;
      }

      float u[8];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
#pragma unroll
        for (int v = 0; v < 4; ++v) u[4 * t + v] = acc[t][v];
      }
      if (tok0 + kTok > vis) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int j = tok0 + 16 * (i >> 2) + 4 * g4 + (i & 3);
          u[i] = j < vis ? u[i] : -INFINITY;
        }
      }
      float mt = fmaxf(fmaxf(fmaxf(u[0], u[1]), fmaxf(u[2], u[3])), fmaxf(fmaxf(u[4], u[5]), fmaxf(u[6], u[7])));
      const float mb = quad_max(mt) * sl2;
      uint32_t pw[4] = {0u, 0u, 0u, 0u};
      float gam = 1.0f;
      if (mb > -INFINITY) {
        const float m_new = fmaxf(m, mb);
        float e[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) e[i] = __builtin_amdgcn_exp2f(fmaf(u[i], sl2, -m_new));
        float esum = ((e[0] + e[1]) + (e[2] + e[3])) + ((e[4] + e[5]) + (e[6] + e[7]));
        esum = quad_sum(esum);
        gam = __builtin_amdgcn_exp2f(m - m_new);
        l = gam * l + esum;
        m = m_new;
#pragma unroll
        for (int i = 0; i < 4; ++i) pw[i] = bf16_bits(e[2 * i]) | (bf16_bits(e[2 * i + 1]) << 16);
      }
      // P of tokens 16t + 4g4 .. +3 at bytes 32t + 8g4 of the row
      uint8_t* prow = xp + (16 * w + n16) * (kTok * 2) + 8 * g4;
      *reinterpret_cast<v2i*>(prow) = v2i{(int)pw[0], (int)pw[1]};
      *reinterpret_cast<v2i*>(prow + 32) = v2i{(int)pw[2], (int)pw[3]};
      if (g4 == 0) *reinterpret_cast<v4f*>(xg + (16 * w + n16) * 4) = v4f{gam, l, m, 0.0f};
      lds_wait();
      if (lane == 0) fstore(xf + w, k + 1);
    }
    barrier_vm_lgkm0<63>();
  } else {
    // =========================== PV waves ====================================
    const int dq = __builtin_amdgcn_readfirstlane(w - 4);
    const int row0 = 64 * g + n, row1 = row0 + 32;
    const uint32_t smem_base = lds_offset(smem);
    // latent copy j of a block: token 8dq + j of the block, lane = LDS chunk, global
    // chunk lane ^ swz(token) (swz of 8dq + j is wave-uniform)
    const uint32_t lane16 = (uint32_t)(lane << 4);
    // RoPE copy: token 8dq + lane/8, LDS chunk lane%8 <- global chunk (lane%8) ^ ((token >> 1) & 7)
    const int rtok = 8 * dq + (lane >> 3);
    const uint32_t rope_v = (uint32_t)((lane >> 3) * (kDr * 2) + (((lane & 7) ^ ((rtok >> 1) & 7)) << 4));

    int ib = cur_b, ib_lo = cur_p0, ib_hi = cur_end;
    auto page_entry = [&](int kb) -> const int32_t* {
      const int gb = gstart + min(kb >> 1, (nblk >> 1) - 1);
      while (gb >= ib_hi) {
        ++ib;
        ib_lo = ib_hi;
        ib_hi = prefix[ib + 1];
      }
      return page_table + (int64_t)ib * a.max_pages + (gb - ib_lo);
    };
    const uint32_t pg_ring = smem_base + kRingBase + 16 * dq;
    const int* pg_ring_p = reinterpret_cast<const int*>(smem + kRingBase + 16 * dq);
    auto request_page = [&](int kb) {
      const int32_t* e = page_entry(kb);
      if (lane == 0) g2lds4_so(reinterpret_cast<const uint8_t*>(e), 0u, pg_ring + 4 * (kb & 3));
    };
    uint32_t stage_bad = 0;
    auto page_ok = [&](int page) { return page >= 0 && page < a.num_pages; };
    auto copy_latent = [&](int kb, int page) {
      const int stg = kb % kLatSt;
      const bool badp = !page_ok(page);
      if (badp) page = 0;
      stage_bad = (stage_bad & ~(1u << stg)) | ((badp ? 1u : 0u) << stg);
      const uint8_t* src = reinterpret_cast<const uint8_t*>(kv_lat) + ((int64_t)page * kPage + kTok * (kb & 1)) * kRowB;
      const uint32_t dst = smem_base + stg * kLatB;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int tok = 8 * dq + j;
        g2lds16_so(src + tok * kRowB, lane16 ^ (uint32_t)(swz(tok) << 4), dst + tok * kRowB);
      }
    };
    auto copy_rope = [&](int kb, int page) {
      if (!page_ok(page)) page = 0;
      const uint8_t* rp = reinterpret_cast<const uint8_t*>(a.k_rope) +
                          ((int64_t)page * kPage + kTok * (kb & 1) + 8 * dq) * (kDr * 2);
      g2lds16_so(rp, rope_v, smem_base + kRopeBase + (kb % kRopeSt) * kRopeB + 1024 * dq);
    };
    // prologue: ids of blocks 0..3 through the scalar cache, ids 4 and 5 requested,
    // latent + RoPE of blocks 0 and 1, latent of block 2
    int pg_rope, pg_lat;
    {
      const int p0 = *page_entry(0);
      const int p1 = *page_entry(1);
      pg_rope = *page_entry(2);
      pg_lat = *page_entry(3);
      request_page(4);
      request_page(5);
      copy_latent(0, p0);
      copy_rope(0, p0);
      copy_latent(1, p1);
      copy_rope(1, p1);
      copy_latent(2, pg_rope);
    }
    v16f O[8];
#pragma unroll
    for (int T = 0; T < 8; ++T) O[T] = v16f{0};
    // transposed reads: read rr (K elements 4rr..4rr+3 of half h) of dim tile T,
    // K-step kk at stage | tr_off[rr] | (kk << 14) ^ (T << 6)
    const int L16 = lane & 15, gq = (lane >> 4) & 3, qq = L16 & 3, kq = L16 >> 2;
    uint32_t tr_off[2];
#pragma unroll
    for (int rr = 0; rr < 2; ++rr) {
      const int tok = 8 * (gq >> 1) + 4 * rr + kq;
      const int chunk = 16 * dq + 2 * (gq & 1) + (qq >> 1);
      tr_off[rr] = (uint32_t)(tok << 10) | (uint32_t)(((chunk ^ swz(tok))) << 4) | (uint32_t)(8 * (qq & 1));
    }
    // top-of-period wait: RoPE of block k followed by the latent of block k+1, the
    // previous period's stores if any and its 10 requests
    auto top_barrier = [&](int k, bool after_stores) {
      if (k + 1 >= nblk) barrier_vm_lgkm0<0>();
      else if (k == 0) barrier_vm_lgkm0<17>();
      else if (after_stores) barrier_vm_lgkm0<18 + kStores>();
      else barrier_vm_lgkm0<18>();
    };

    v2i rv[4][2][2];
    v4i P0[2], P1[2];
    v4f gl0, gl1;
    bool cur_bad = false, stored = false;
    for (int k = 0;; ++k) {
      top_barrier(k, stored);
      stored = false;
      if (k > 0) {
        // ---- PV of block k-1 ------------------------------------------------
#pragma unroll
        for (int T = 0; T < 4; ++T) {
          O[2 * T] *= gl0[0];
          O[2 * T + 1] *= gl1[0];
        }
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
          for (int T = 0; T < 4; ++T) {
            const v4i A = v4i{rv[T][kk][0][0], rv[T][kk][0][1], rv[T][kk][1][0], rv[T][kk][1][1]};
            O[2 * T] = mfma_bf16_32x32x16(A, P0[kk], O[2 * T]);
            O[2 * T + 1] = mfma_bf16_32x32x16(A, P1[kk], O[2 * T + 1]);
          }
        }
        if (k == nblk || ((k & 1) == 0 && gstart + (k >> 1) >= cur_end)) {
          // the piece ends: exactly kStores stores (the next top-of-period wait counts them)
          const int64_t pid = a.chunk_blocks == 0 ? (int64_t)unit + cur_b
                                                  : (int64_t)cur_b * a.num_splits + cur_blk0 / a.chunk_blocks;
          const bool whole = cur_blk0 == 0 && gstart + (k >> 1) >= cur_end;   // the piece is its whole sequence
          float inv[2], lse[2];
#pragma unroll
          for (int r = 0; r < 2; ++r) {
            const v4f gl = r == 0 ? gl0 : gl1;
            const float lfin = gl[1];
            const bool empty = !(lfin > 0.0f);
            inv[r] = empty ? 0.0f : 1.0f / lfin;
            lse[r] = empty ? -INFINITY : (gl[2] + log2f(lfin)) * kLn2f;
            if (cur_bad) {
              inv[r] = __builtin_nanf("");
              lse[r] = __builtin_nanf("");
            }
          }
          store_piece(a, O, inv[0], inv[1], lse[0], lse[1], row0, row1, dq, h, pid, cur_b, whole);
#pragma unroll
          for (int T = 0; T < 8; ++T) O[T] = v16f{0};
          stored = true;
        }
      }
      if (k + 2 < nblk) {
        request_page(k + 6);
        copy_rope(k + 2, pg_rope);
        copy_latent(k + 3, pg_lat);
        pg_rope = pg_lat;                            // the RoPE copy of the next period is block k+3
      }
      if (k == nblk) break;

      // ---- block k: bookkeeping, V^T tiles, codes and state ---------------------
      const int gb = gstart + (k >> 1), hk = k & 1;
      if (gb >= cur_end) {
        enter_piece(gb);
        cur_bad = false;
      }
      cur_bad |= ((stage_bad >> (k % kLatSt)) & 1u) != 0;
      const int valid = max(0, min(kTok, cur_n - ((gb - cur_p0) * kPage + kTok * hk)));
      if (valid < kTok) {
        // slots past the sequence end: clear the bytes this wave reads (stale data could hold NaN; P is 0 there)
        uint8_t* stp = smem + (k % kLatSt) * kLatB;
        const int nz = (kTok - valid) * 16;
        for (int i = lane; i < nz; i += 64) {
          const int t = valid + (i >> 4);
          const int c = 16 * dq + (i & 15);
          *reinterpret_cast<v4i*>(stp + t * kRowB + ((c ^ swz(t)) << 4)) = v4i{0, 0, 0, 0};
        }
      }
      const uint32_t st_lds = smem_base + (k % kLatSt) * kLatB;
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
        for (int T = 0; T < 4; ++T) {
#pragma unroll
          for (int rr = 0; rr < 2; ++rr)
            rv[T][kk][rr] = lds_read_tr16_at(st_lds + ((tr_off[rr] | (uint32_t)(kk << 14)) ^ (uint32_t)(T << 6)));
        }
      }
      {
        // one exit for both ends of the wait, decided again from the last poll: codes
        // never published, or a zero bound, mark the piece, which then comes out NaN
        v4i f4;
        int spin = 0;
        do {
          f4 = fload4(xf);
        } while (!(f4[0] > k && f4[1] > k && f4[2] > k && f4[3] > k) && ++spin < a.spin_limit);
        if (!(f4[0] > k && f4[1] > k && f4[2] > k && f4[3] > k) || a.spin_limit <= 0) cur_bad = true;
      }
      asm volatile("" ::: "memory");
      gl0 = *reinterpret_cast<const v4f*>(xg + n * 4);
      gl1 = *reinterpret_cast<const v4f*>(xg + (n + 32) * 4);
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        P0[kk] = *reinterpret_cast<const v4i*>(xp + n * (kTok * 2) + 32 * kk + 16 * h);
        P1[kk] = *reinterpret_cast<const v4i*>(xp + (n + 32) * (kTok * 2) + 32 * kk + 16 * h);
      }
      const int pg_next = pg_ring_p[(k + 4) & 3];
      lds_wait();
      pg_lat = __builtin_amdgcn_readfirstlane(pg_next);
    }
  }
}

// The step's new tokens into the BF16 cache: row copies, one wave per token.
__global__ __launch_bounds__(256) void append_bf16_kernel(const uint16_t* __restrict__ c_kv_new,
                                                          const uint16_t* __restrict__ k_rope_new,
                                                          const int32_t* __restrict__ page_table,
                                                          const int32_t* __restrict__ seq_lens, int B, int n_new,
                                                          int max_pages, int num_pages, uint16_t* __restrict__ kv_latent,
                                                          uint16_t* __restrict__ k_rope) {
  const int lane = threadIdx.x & 63;
  const int64_t tok = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (tok >= (int64_t)B * n_new) return;
  const int b = (int)(tok / n_new), t = (int)(tok % n_new);
  const int pos = seq_lens[b] - n_new + t;
  if (pos < 0 || pos >= max_pages * kPage) return;
  const int page = page_table[(int64_t)b * max_pages + pos / kPage];
  if (page < 0 || page >= num_pages) return;
  const int64_t slot = (int64_t)page * kPage + (pos % kPage);
  reinterpret_cast<uint4*>(kv_latent + slot * kDc)[lane] = reinterpret_cast<const uint4*>(c_kv_new + tok * kDc)[lane];
  if (lane < 8)
    reinterpret_cast<uint4*>(k_rope + slot * kDr)[lane] = reinterpret_cast<const uint4*>(k_rope_new + tok * kDr)[lane];
}

}  // namespace

hipError_t launch_append_bf16(const uint16_t* c_kv_new, const uint16_t* k_rope_new, const int32_t* page_table,
                              const int32_t* seq_lens, int B, int n_new, int max_pages, int num_pages,
                              uint16_t* kv_latent, uint16_t* k_rope, hipStream_t stream) {
  const int64_t toks = (int64_t)B * n_new;
  if (toks == 0) return hipSuccess;
  hipLaunchKernelGGL(append_bf16_kernel, dim3((unsigned)((toks + 3) / 4)), dim3(256), 0, stream, c_kv_new,
                     k_rope_new, page_table, seq_lens, B, n_new, max_pages, num_pages, kv_latent, k_rope);
  return hipGetLastError();
}

hipError_t launch_decode_bf16(const DecodeArgs& a, const uint16_t* kv_lat, hipStream_t stream) {
  const int units = a.chunk_blocks == 0 ? a.num_splits : a.B * a.num_splits;
  if (units <= 0) return hipSuccess;
  const int64_t grid = (int64_t)((units + 7) / 8) * 8 * a.G;
  if (grid > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL(decode_bf16_kernel, dim3((unsigned)grid), dim3(512), 0, stream, a, kv_lat, a.prefix,
                     a.page_table, a.seq_lens);
  return hipGetLastError();
}

}  // namespace snapmla
