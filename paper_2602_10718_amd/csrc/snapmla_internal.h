// Host-side launch interfaces between the C ABI (api.hip) and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace snapmla {

// Workspace carve-up shared by decode and combine.
struct WsLayout {
  int R = 0, G = 0, rows_pad = 0, pieces = 0;
  int units = 0;
  int pad = 0;              // balanced plan: virtual blocks charged to each sequence start
  size_t q8 = 0, sq = 0, prefix = 0, flags = 0, zero = 0, ctrl = 0, desc = 0, lse = 0, o = 0, total = 0;
};
WsLayout ws_layout(int B, int q_len, int H, int num_splits, int kv_chunk_tokens);

// Balanced plan: part u covers the real blocks of the virtual block positions
// [u*TV/W, (u+1)*TV/W), TV = T + pad*B, where sequence b occupies the virtual positions
// [prefix[b] + pad*b, prefix[b+1] + pad*(b+1)) with its pad leading positions empty.
// A part that holds a sequence start so gets up to pad fewer blocks: a range that
// crosses into another sequence pays a piece end and a piece start mid-range (~2.7
// blocks' time with one row group).  With several row groups the period is the waves'
// own work and equal block counts are kept (pad 0).
constexpr int kPlanPad = 4;
// units up to which the prep kernel maps units to sequences through an LDS table
constexpr int kPlanTable = 1024;

struct PrepArgs {
  const uint16_t* q_nope;   // [B*R][512]
  uint8_t* q8;              // [B*R][512]
  float* sq;                // [B*R]
  int64_t rows;             // B*R
  const int32_t* seq_lens;
  int32_t* prefix;          // [B+1] cumulative 64-token block counts of valid sequences
  int32_t* flags;           // [B] 1 = sequence rejected (data error)
  uint8_t* zero;            // 1 KiB that the decode kernel reads in place of slots past a sequence end
  int32_t* desc;            // [units][kDescInts] start descriptor of each split unit (see kDesc*)
  int B, q_len, max_pages, chunk_blocks, num_splits, units;
  int pad = 0;              // balanced plan's virtual blocks per sequence start (WsLayout::pad)
  // Final results written by the decode itself (out != nullptr): the rows of sequences
  // without blocks (empty: o = 0, LSE = -inf; rejected by a data error: NaN), written by
  // the row waves, and ctrl[0] = 1, which tells the combine that the decode also wrote
  // every sequence one piece covers (ctrl[0] = 0 when out is null: partials only).
  int32_t* ctrl = nullptr;
  void* out = nullptr;              // [B*R][512] bf16 (out_dtype 0) or f32 (1)
  float* out_lse = nullptr;         // [B*R] or null
  int out_dtype = 0, R = 0;
  bool quantize = true;             // the row waves quantize the queries (FP8 cache) or only
                                    // write the rows of sequences without blocks
  // optional fused quantize-on-append of n_new tokens per sequence (ablocks workgroups of
  // four tokens; none when ablocks == 0), run beside the query quantization
  const uint16_t* c_kv_new = nullptr;   // [B][n_new][512]
  const uint16_t* k_rope_new = nullptr; // [B][n_new][64]
  const int32_t* page_table = nullptr;
  uint8_t* kv_latent = nullptr;
  float* kv_scale = nullptr;
  uint16_t* k_rope = nullptr;
  int n_new = 0, num_pages = 0, ablocks = 0;
};

// Start descriptor of a split unit (a workgroup's range of 64-token blocks), written
// by the prep kernel so that a workgroup begins without searching the plan:
constexpr int kDescInts = 8;
constexpr int kDescStart = 0;    // first global block of the range
constexpr int kDescEnd = 1;      // one past the last (start >= end: nothing to do)
constexpr int kDescSeq = 2;      // sequence of the first block
constexpr int kDescP0 = 3;       // its first global block (prefix[seq])
constexpr int kDescP1 = 4;       // one past its last (prefix[seq + 1])
constexpr int kDescLen = 5;      // its length in tokens

constexpr int kDefaultSpinLimit = 1 << 22;
// process-wide spin limit of the decode launches (snapmla_debug_set_spin_limit)
int spin_limit();

struct DecodeArgs {
  const uint16_t* q_nope;   // [B*R][512] bf16 (read by the BF16-cache kernel only)
  const uint8_t* q8;
  const float* sq;
  const uint16_t* q_rope;   // [B*R][64]
  const uint8_t* kv_latent;
  const float* kv_scale;
  const uint16_t* k_rope;
  const int32_t* page_table;
  const int32_t* seq_lens;
  const int32_t* prefix;
  const int32_t* desc;      // [units][kDescInts]
  const uint8_t* zero;
  float* part_o;            // [pieces][rows_pad * 512]: rows, or part_tile_offset order (rows_pad > 64)
  float* part_lse;          // [pieces][rows_pad]
  int B, q_len, H, R, G, rows_pad, max_pages, num_pages, causal;
  int num_splits, chunk_blocks;  // chunk_blocks == 0: balanced plan over num_splits parts
  float sl2;                     // softmax scale * log2(e)
  // Upper bound on the polls of each handshake wait inside the decode kernels.  The
  // waits end by construction (every flag they poll is stored once per block, before
  // its owner waits on anything); the bound only guarantees termination.  A wait that
  // reaches it marks its piece, whose outputs and LSEs then come out NaN.
  int spin_limit = kDefaultSpinLimit;
  // QK content product with exact float32 accumulation (F16 MFMA on the exactly
  // converted E4M3 codes) instead of the FP8 MFMA
  int qk_exact = 0;
  // Direct results (out != nullptr): a piece that covers its whole sequence writes the
  // final rows and LSEs there instead of a partial (the one-piece merge is exact).
  void* out = nullptr;              // [B*R][512] bf16 (out_dtype 0) or f32 (1)
  float* out_lse = nullptr;         // [B*R] or null
  int out_dtype = 0;
};

// Validity of a sequence's length (the data errors of the decode): true when the
// length is usable, i.e. 0, or q_len .. max_pages*64 tokens (and, with fixed chunks,
// at most num_splits chunks).  Shared by the plan and the rows of rejected sequences.
__host__ __device__ inline bool seq_len_ok(int n, int q_len, int max_pages, int chunk_blocks, int num_splits) {
  bool ok = (n == 0) || (n >= q_len && (int64_t)n <= (int64_t)max_pages * 64);
  if (ok && chunk_blocks > 0) ok = ((n + 63) / 64 + chunk_blocks - 1) / chunk_blocks <= num_splits;
  return ok;
}

// Float32 offset of a partial-output element inside its piece's slot when the rows
// form several 64-row groups (rows_pad > 64).  The order follows the PV waves'
// accumulator tiles, so that each 16-byte store instruction of a wave writes 1 KiB of
// consecutive memory: row group g (rows 64g..64g+63), dimension quarter dq (128
// dimensions), row tile rt (32 rows), dimension tile T (32 dimensions), chunk pair q
// (8 dimensions), then lane n + 32h, which holds row 64g + 32rt + n, dimensions
// 128dq + 32T + 8q + 4h .. +3.  With one row group the slot keeps plain rows
// ([64][512]): there the merge skips, row by row, the pieces whose weight underflows
// to zero, which needs each row's partial in its own cache lines.
__host__ __device__ constexpr int64_t part_tile_offset(int g, int dq, int rt, int T, int q, int lane) {
  return (int64_t)g * 32768 + dq * 8192 + rt * 4096 + T * 1024 + q * 256 + lane * 4;
}

struct CombineArgs {
  const float* part_o;
  const float* part_lse;
  const int32_t* prefix;
  const int32_t* flags;
  const int32_t* ctrl;      // ctrl[0] == 1: sequences with at most one piece are final already
  const int32_t* seq_lens;
  void* out;
  float* lse;
  int B, q_len, H, R, rows_pad, num_splits, chunk_blocks, out_dtype;
  int pad;                  // balanced plan's virtual blocks per sequence start (WsLayout::pad)
};

struct FetchArgs {
  const uint8_t* kv_latent;   // [num_pages][64][512]
  const float* kv_scale;      // [num_pages][64]
  const uint16_t* k_rope;     // [num_pages][64][64]
  const int32_t* page_table;  // [B][max_pages]
  const int32_t* cu;          // [B+1] output row offsets; sequence b has cu[b+1] - cu[b] tokens
  uint16_t* out;              // [cu[B]][576] bf16
  int B, max_pages, num_pages;
};

hipError_t launch_quantize_rows(const uint16_t* x, int64_t rows, uint8_t* codes, float* scale,
                                hipStream_t stream);
hipError_t launch_append(const uint16_t* c_kv_new, const uint16_t* k_rope_new, const int32_t* page_table,
                         const int32_t* seq_lens, int B, int n_new, int max_pages, int num_pages,
                         uint8_t* kv_latent, float* kv_scale, uint16_t* k_rope, hipStream_t stream);
hipError_t launch_encode(const float* x, int64_t n, uint8_t* codes, hipStream_t stream);
hipError_t launch_prep(const PrepArgs& a, hipStream_t stream);
hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream);
hipError_t launch_combine(const CombineArgs& a, hipStream_t stream);
hipError_t launch_fetch_dequant(const FetchArgs& a, hipStream_t stream);
hipError_t launch_decode_bf16(const DecodeArgs& a, const uint16_t* kv_latent_bf16, hipStream_t stream);
hipError_t launch_append_bf16(const uint16_t* c_kv_new, const uint16_t* k_rope_new, const int32_t* page_table,
                              const int32_t* seq_lens, int B, int n_new, int max_pages, int num_pages,
                              uint16_t* kv_latent, uint16_t* k_rope, hipStream_t stream);
hipError_t launch_quantize_cache_config(const uint16_t* c_kv, const uint16_t* k_rope, const int32_t* page_table,
                                        const int32_t* cu, int B, int max_pages, int num_pages, int config,
                                        uint32_t* amax_word, uint8_t* kv_latent, float* kv_scale,
                                        uint16_t* k_rope_out, hipStream_t stream);

// One FP8 16x16x128 MFMA per 16x128 tile pair (test hook of the QK content term).
hipError_t launch_mfma_fp8(const uint8_t* a, const uint8_t* b, float* c, int64_t tiles, hipStream_t stream);

// Read-stream ceiling (measurement): the pages of nblk blocks streamed into LDS.
constexpr int kCeilingMaxBlocks = 1792;   // blocks per workgroup (their page ids sit in LDS)
struct CeilingArgs {
  const uint8_t* kv_latent;
  const float* kv_scale;
  const uint16_t* k_rope;
  const int32_t* pages;     // [nblk] physical page of each block, in stream order
  uint32_t* out;            // [units] per-workgroup checksum
  int nblk, num_pages, units;
};
hipError_t launch_read_ceiling(const CeilingArgs& a, hipStream_t stream);
// Plain read stream (measurement): n16 16-byte words read by `grid` workgroups of 256 threads.
hipError_t launch_read_stream(const void* buf, int64_t n16, int grid, uint32_t* out, hipStream_t stream);

}  // namespace snapmla
