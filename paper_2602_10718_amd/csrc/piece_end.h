// Piece-end results of one PV wave of the decode kernels (Algorithm 1 finalisation:
// o = O / l and the log-sum-exp of each row).
#pragma once

#include "snapmla_device.h"
#include "snapmla_internal.h"

namespace snapmla {

// Store instructions of one PV wave at the end of a piece: 2 row tiles x (16 output
// chunks + 1 log-sum-exp).  The top-of-period waits that follow count them, so every
// destination below takes exactly this many.
constexpr int kPieceStores = 2 * (16 + 1);

__device__ __forceinline__ uint32_t f32_to_bf16_bits(float x) {
  const uint32_t u = __float_as_uint(x);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;     // NaN stays NaN
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;           // round to nearest even
}

// The PV wave that owns latent dimensions 128dq..128dq+127 holds, for row tile r
// (query row row_r of the sequence), O^T tile T in O[2T + r]: element v of a lane
// (half h) is dimension 128dq + 32T + 8(v/4) + 4h + v%4.  inv_r = 1/l (0 for a row
// without tokens, NaN for a rejected piece), lse_r its log-sum-exp.
//
// A piece that covers its whole sequence (whole, with a.out set) is final: its rows
// go to out[seq*R + row] in the output type and its LSEs to out_lse; otherwise the
// normalized partial and its LSE go to the piece's slot pid of the workspace, which
// snapmla_combine merges.  With several row groups the slot is in accumulator tile
// order (part_tile_offset: each store instruction writes 1 KiB of consecutive bytes),
// with one it holds plain rows (32 bytes in each of 32 rows per instruction).  Rows
// from R up to rows_pad (padding of the last row group) always go to the slot, which
// holds rows_pad rows and is never read for them: the store count stays the same
// whatever the destination.
__device__ __forceinline__ void store_piece(const DecodeArgs& a, const v16f (&O)[8], float inv0, float inv1,
                                            float lse0, float lse1, int row0, int row1, int dq, int h,
                                            int64_t pid, int seq, bool whole) {
  const bool direct = whole && a.out != nullptr;
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int row = r == 0 ? row0 : row1;
    const float inv = r == 0 ? inv0 : inv1;
    const bool tiles = a.rows_pad > 64;
    float* slot = tiles ? a.part_o + pid * a.rows_pad * kDc + part_tile_offset(row >> 6, dq, r, 0, 0, (row & 31) + 32 * h)
                        : a.part_o + (pid * a.rows_pad + row) * kDc + 128 * dq + 4 * h;
    float* slot_lse = a.part_lse + pid * a.rows_pad + row;
    // float offsets of tile T, chunk pair q inside the slot (plain rows: 32T + 8q)
    const int st = tiles ? 1024 : 32, sq = tiles ? 256 : 8;
    const bool mine = direct && row < a.R;
    const int64_t orow = (int64_t)seq * a.R + row;
    if (direct && a.out_dtype == 0) {
      // bf16 rows: four values (8 bytes) per store
      // (a padding row writes its bf16 pairs into the first half of its slot cells)
      uint16_t* dst = mine ? static_cast<uint16_t*>(a.out) + orow * kDc + 128 * dq + 4 * h
                           : reinterpret_cast<uint16_t*>(slot);
      const int bt = mine ? 32 : 2 * st, bq = mine ? 8 : 2 * sq;        // uint16 units
#pragma unroll
      for (int T = 0; T < 4; ++T) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const v16f& o = O[2 * T + r];
          const uint32_t lo = f32_to_bf16_bits(o[4 * q + 0] * inv) | (f32_to_bf16_bits(o[4 * q + 1] * inv) << 16);
          const uint32_t hi = f32_to_bf16_bits(o[4 * q + 2] * inv) | (f32_to_bf16_bits(o[4 * q + 3] * inv) << 16);
          *reinterpret_cast<v2i*>(dst + bt * T + bq * q) = v2i{(int)lo, (int)hi};
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    } else {
      // float32 rows (final or partial): four values (16 bytes) per store
      float* dst = mine ? static_cast<float*>(a.out) + orow * kDc + 128 * dq + 4 * h : slot;
      const int ft = mine ? 32 : st, fq = mine ? 8 : sq;
#pragma unroll
      for (int T = 0; T < 4; ++T) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const v16f& o = O[2 * T + r];
          *reinterpret_cast<v4f*>(dst + ft * T + fq * q) =
              v4f{o[4 * q + 0] * inv, o[4 * q + 1] * inv, o[4 * q + 2] * inv, o[4 * q + 3] * inv};
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    if (h == 0) {
      float* ldst = (mine && a.out_lse != nullptr) ? a.out_lse + orow : slot_lse;
      *ldst = r == 0 ? lse0 : lse1;
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

}  // namespace snapmla
