/*
 * snapmla.h -- C ABI of libsnapmla.so: FP8 Multi-head Latent Attention decode
 * over a paged, per-token-quantized KV cache, for AMD Instinct MI355X (gfx950).
 *
 * The method is SnapMLA (arXiv 2602.10718):
 *   - RoPE-aware per-token KV quantization (Section 3.1): the 512-d content
 *     latent c_KV of every token is stored as OCP FP8 E4M3 with one float32
 *     scale per token; the 64-d RoPE key stays BF16.
 *   - Quantized PV pipeline reconstruction (Section 3.2, Appendix D): the
 *     per-token V scale is fused into the probabilities, each 64-token block of
 *     fused probabilities is quantized to E4M3 with its own dynamic scale, and
 *     the online-softmax state is kept in the current block-scale domain
 *     ("implicit dequantization").
 *   - Fused token preparation (Section 3.3, Layer 1): quantize-on-append writes
 *     new tokens straight into their paged slots; query quantization is fused
 *     into the decode call.
 * The split-KV log-sum-exp merge (snapmla_combine) uses the per-row
 * log-sum-exp that Algorithm 1 returns next to the output.
 *
 * Conventions for every function:
 *   - Every pointer argument is DEVICE memory owned by the caller unless noted;
 *     the library allocates nothing and keeps no state besides a cached device
 *     property record.  page_table, seq_lens and lse need 4-byte alignment;
 *     every other pointer must be 16-byte aligned (SNAPMLA_MISALIGNED otherwise).
 *   - Work is enqueued on `stream` (a hipStream_t; 0 is the legacy default
 *     stream); calls return before the work runs.  Calls are thread-safe.
 *   - The return value is a status code (SNAPMLA_OK == 0).  On failure nothing
 *     is enqueued and snapmla_get_last_error() returns a message (thread-local).
 *   - Data errors that need device data to detect (a page id outside
 *     [0, num_pages), a sequence longer than max_pages * 64, or
 *     0 < seq_len < q_len) never cause an out-of-bounds access: decode writes
 *     NaN into every output row of that sequence and quantize_append skips the
 *     token.
 *
 * Cache planes (one page = 64 consecutive tokens of one sequence):
 *   kv_latent  uint8  [num_pages][64][512]   E4M3 codes of c_KV (also the value operand)
 *   kv_scale   float  [num_pages][64]        per-token scale sigma_K (row = sigma_K * E4M3 codes)
 *   k_rope     bf16   [num_pages][64][64]    RoPE key, stored unscaled (bit copy of the input)
 *   page_table int32  [B][max_pages]         physical page of each 64-token logical page
 *   seq_lens   int32  [B]                    tokens in the cache per sequence, INCLUDING the
 *                                            tokens of the current step
 * Queries:
 *   q_nope  bf16 [B][q_len][H][512]   absorbed query content part (q^C W^UK, Section 2)
 *   q_rope  bf16 [B][q_len][H][64]
 * A "row" is one (query token t, head h) pair, row index t*H + h; a sequence
 * has R = q_len*H rows.  With causal != 0 row t attends to the first
 * seq_len - q_len + 1 + t tokens; otherwise every row attends to all seq_len.
 */
#ifndef SNAPMLA_H
#define SNAPMLA_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SNAPMLA_ABI_VERSION 3

enum snapmla_status {
  SNAPMLA_OK = 0,
  SNAPMLA_INVALID_ARGUMENT = 1,   /* a size, pointer or flag is out of range */
  SNAPMLA_UNSUPPORTED = 2,        /* valid but not implemented (e.g. page_size != 64) */
  SNAPMLA_WORKSPACE_TOO_SMALL = 3,
  SNAPMLA_MISALIGNED = 4,         /* a pointer is not 16-byte aligned */
  SNAPMLA_HIP_ERROR = 5           /* a HIP runtime call failed */
};

/* Flags of snapmla_decode and snapmla_append_decode. */
enum snapmla_decode_flags {
  /* Form the content term <q8, c8> with exact float32 accumulation: the E4M3
   * codes are converted to f16 (an exact conversion) and multiplied with the F16
   * matrix cores.  Without it the FP8 matrix cores sum each group of eight
   * consecutive products with every product truncated to a multiple of
   * 2^(E-13), E the group's largest exponent sum (gfx950 behaviour, measured
   * bit for bit), which moves logits in the thousands by up to ~1e-1 and the
   * LSE with them.  Same inputs, outputs and workspace; slower (the conversion
   * and twice the matrix-core work of the content term). */
  SNAPMLA_DECODE_EXACT_QK = 1
};

/* ABI version of the loaded library (SNAPMLA_ABI_VERSION). */
int snapmla_abi_version(void);

/* Message for the last failed call on this thread ("" if none).  The pointer
 * stays valid until the next call on the same thread. */
const char* snapmla_get_last_error(void);

/*
 * snapmla_quantize_append -- fused quantize-on-append (Section 3.3, Layer 1,
 * Fused-K-Append; per-token granularity of Section 3.1 and Appendix C).
 *
 * For every sequence b and new token t < n_new, the token is written at
 * position pos = seq_lens[b] - n_new + t of sequence b, i.e. into page
 * page_table[b][pos / 64], slot pos % 64.  The latent row x (512 bf16) is
 * quantized per token:
 *     a = max_i |x_i|;  sigma = max(fp32(a / 448), 2^-40);  code_i = E4M3_rne(fp32(x_i / sigma))
 * with IEEE float32 divisions, and sigma goes to kv_scale.  The RoPE row is
 * copied bit for bit.  Tokens whose position is negative, beyond
 * max_pages * 64, or whose page id is outside [0, num_pages) are skipped.
 *
 *   c_kv_new    bf16 [B][n_new][512]   device, read
 *   k_rope_new  bf16 [B][n_new][64]    device, read
 *   page_table  int32 [B][max_pages]   device, read
 *   seq_lens    int32 [B]              device, read (already counting the new tokens)
 *   page_size   must be 64 (SNAPMLA_UNSUPPORTED otherwise)
 *   kv_latent, kv_scale, k_rope        device cache planes, written at the new slots only
 * B >= 0, n_new >= 0 (B*n_new == 0 enqueues nothing), max_pages >= 1, num_pages >= 1.
 */
int snapmla_quantize_append(const void* c_kv_new, const void* k_rope_new,
                            const int32_t* page_table, const int32_t* seq_lens,
                            int32_t B, int32_t n_new, int32_t max_pages, int32_t num_pages,
                            int32_t page_size,
                            uint8_t* kv_latent, float* kv_scale, void* k_rope,
                            hipStream_t stream);

/*
 * snapmla_quantize_rows -- the same per-row quantizer as above, dense: rows
 * x[r][0..511] (bf16) -> codes[r][0..511] (E4M3) and scale[r] (float32).
 * snapmla_decode applies it to q_nope (Section 3.3, Fused-Q-Quant; one query
 * scale per row, Algorithm 1's sigma_q).  rows >= 0.
 */
int snapmla_quantize_rows(const void* x, int64_t rows, uint8_t* codes, float* scale,
                          hipStream_t stream);

/*
 * Workspace for snapmla_decode / snapmla_combine, in bytes.  It holds the
 * quantized queries, the split plan and, per KV piece, a float32 partial
 * output of 64*ceil(R/64) rows x 512 (in an order of the library's own, read
 * only by snapmla_combine) and partial log-sum-exp.
 *   kv_chunk_tokens == 0: balanced split over `num_splits` parts of the total
 *                         64-token block count (num_splits >= 1; a sequence
 *                         may span several parts and a part several sequences;
 *                         with R <= 64 each sequence start counts as 4 extra
 *                         blocks, so parts that hold a sequence boundary get
 *                         up to 4 fewer blocks)
 *   kv_chunk_tokens  > 0: every sequence is cut into chunks of kv_chunk_tokens
 *                         (a multiple of 64); num_splits bounds the chunks per
 *                         sequence (sequences needing more are flagged NaN).
 *                         With kv_chunk_tokens >= max_pages*64 and num_splits == 1
 *                         no sequence is split (the unsplit plan: one piece per
 *                         sequence, no snapmla_combine needed when out is given)
 * *bytes receives the size; returns SNAPMLA_INVALID_ARGUMENT on bad sizes.
 */
int snapmla_decode_workspace_size(int32_t B, int32_t q_len, int32_t H,
                                  int32_t num_splits, int32_t kv_chunk_tokens,
                                  size_t* bytes);

/*
 * snapmla_decode -- FP8 MLA decode over the paged cache (Algorithm 1 and
 * Appendix D; Section 2 absorbed score).  Enqueues the query quantization and
 * the decode kernel.
 *
 * Per row r and cached token j the restored logit is
 *     s = softmax_scale * ( sigma_q[r] * sigma_K[j] * <q8_r, c8_j> + <q_rope_r, k_rope_j> )
 * (FP8 x FP8 content term, BF16 x BF16 RoPE term, both accumulated in float32).
 * The tokens are visited in 64-token blocks in increasing order; per block:
 * online softmax with running max m, e = exp(s - m); fused probabilities
 * p' = e * sigma_K; block scale sigma_P = max(max p' / 448, 2^-40);
 * codes pi = E4M3(p' / sigma_P); output and normalizer kept in the sigma_P
 * domain (Appendix D recurrences); the PV product pi x c8 runs in FP8.
 * A KV piece (a sequence's blocks inside one part or chunk of the split plan,
 * see snapmla_decode_workspace_size) that covers its whole sequence writes the
 * final rows o = O / l and LSE = m + ln(sigma_P l) (Algorithm 1 finalisation)
 * into out and lse; the rows of sequences without blocks are written too (o = 0
 * and LSE = -inf when empty, NaN when a data error rejects the sequence).  Every
 * other piece writes its normalized partial output and log-sum-exp into the
 * workspace, and snapmla_combine (same workspace, plan, out, out_dtype and lse)
 * merges them into the remaining rows.  With out == NULL every piece writes a
 * partial and snapmla_combine writes every row.
 *
 *   q_nope, q_rope        bf16 queries (layout above), device, read
 *   kv_latent, kv_scale, k_rope, page_table, seq_lens   cache (layout above), device, read
 *   B >= 0; q_len in {1, 2}; H >= 1 with q_len*H <= 256
 *   max_pages >= 1, num_pages >= 1, page_size == 64
 *   softmax_scale         finite, > 0
 *   causal                0 or 1 (only meaningful for q_len = 2)
 *   num_splits, kv_chunk_tokens   split plan (see snapmla_decode_workspace_size)
 *   flags                 0 or SNAPMLA_DECODE_EXACT_QK (other bits: SNAPMLA_INVALID_ARGUMENT)
 *   workspace / workspace_bytes   device scratch of at least the queried size
 *   out        [B][q_len][H][512], bf16 (out_dtype 0, round to nearest even) or
 *              float32 (1), written; or NULL (partials only)
 *   lse        float32 [B][q_len][H], written; may be NULL (must be NULL when out is)
 */
int snapmla_decode(const void* q_nope, const void* q_rope,
                   const uint8_t* kv_latent, const float* kv_scale, const void* k_rope,
                   const int32_t* page_table, const int32_t* seq_lens,
                   int32_t B, int32_t q_len, int32_t H,
                   int32_t max_pages, int32_t num_pages, int32_t page_size,
                   float softmax_scale, int32_t causal,
                   int32_t num_splits, int32_t kv_chunk_tokens, int32_t flags,
                   void* workspace, size_t workspace_bytes,
                   void* out, int32_t out_dtype, float* lse,
                   hipStream_t stream);

/*
 * snapmla_append_decode -- snapmla_quantize_append of the step's n_new tokens
 * per sequence followed by snapmla_decode, with the quantize-on-append run in
 * the same preparation launch as the query quantization (Section 3.3, Layer 1
 * fuses both token preparations ahead of the attention kernel).  The result,
 * the cache bytes written and the error behaviour are those of the two calls in
 * sequence on `stream`; one kernel launch fewer.
 *   c_kv_new bf16 [B][n_new][512], k_rope_new bf16 [B][n_new][64]   device, read;
 *            token t of sequence b goes to position seq_lens[b] - n_new + t
 *            (n_new == 0: no append, the pointers may be NULL)
 *   kv_latent, kv_scale, k_rope   cache planes, written at the new tokens' slots
 *            and then read by the decode
 *   every other argument as snapmla_decode
 */
int snapmla_append_decode(const void* c_kv_new, const void* k_rope_new, int32_t n_new,
                          const void* q_nope, const void* q_rope,
                          uint8_t* kv_latent, float* kv_scale, void* k_rope,
                          const int32_t* page_table, const int32_t* seq_lens,
                          int32_t B, int32_t q_len, int32_t H,
                          int32_t max_pages, int32_t num_pages, int32_t page_size,
                          float softmax_scale, int32_t causal,
                          int32_t num_splits, int32_t kv_chunk_tokens, int32_t flags,
                          void* workspace, size_t workspace_bytes,
                          void* out, int32_t out_dtype, float* lse,
                          hipStream_t stream);

/* Bytes of the static scratch of snapmla_append_decode_noalloc (128 MiB per GPU). */
#define SNAPMLA_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)

/*
 * snapmla_append_decode_noalloc -- for callers that cannot allocate device memory
 * (code under HIP graph capture, serving loops or harnesses that forbid
 * hipMalloc): the whole step of snapmla_append_decode followed by
 * snapmla_combine, with the workspace in a static array inside the library
 * instead of a caller buffer.  Same results as those two calls with a caller
 * workspace, bit for bit; allocates nothing (the array is part of the library's
 * device code: every GPU the library runs on holds its own 128 MiB copy until
 * the process ends; its device address is looked up once per device, on the
 * first call with that device current).
 *   arguments as snapmla_append_decode, without workspace/workspace_bytes
 *   (out must not be NULL)
 *   the plan's workspace (snapmla_decode_workspace_size) must fit in
 *   SNAPMLA_NOALLOC_SCRATCH_BYTES, else SNAPMLA_WORKSPACE_TOO_SMALL and nothing
 *   is enqueued (a 64-row group per 256 split parts needs ~40 MiB)
 * Every call on one GPU uses that GPU's one array, and nothing in it is assumed
 * to start at zero (each call writes what it reads).  Calls that overlap on one
 * GPU (other streams, other threads, without ordering between them) race on the
 * array and give wrong results: order them on one stream or with events.
 */
int snapmla_append_decode_noalloc(const void* c_kv_new, const void* k_rope_new, int32_t n_new,
                                  const void* q_nope, const void* q_rope,
                                  uint8_t* kv_latent, float* kv_scale, void* k_rope,
                                  const int32_t* page_table, const int32_t* seq_lens,
                                  int32_t B, int32_t q_len, int32_t H,
                                  int32_t max_pages, int32_t num_pages, int32_t page_size,
                                  float softmax_scale, int32_t causal,
                                  int32_t num_splits, int32_t kv_chunk_tokens, int32_t flags,
                                  void* out, int32_t out_dtype, float* lse,
                                  hipStream_t stream);

/*
 * snapmla_decode_bf16 -- the BF16-cache baseline of the paper's comparison
 * (Section 4: the FP8 kernel against MLA decode over a BF16 cache).  Same
 * queries, page table, split plan, workspace and combine as snapmla_decode; the
 * cache holds bf16 latent rows and no scales:
 *   kv_latent bf16 [num_pages][64][512], k_rope bf16 [num_pages][64][64]
 * Per row: s = softmax_scale * (q_nope . c + q_rope . k_rope) in float32 (BF16
 * MFMA), online softmax over 32-token blocks, P rounded to bf16 for the BF16 PV
 * product (the normalizer sums the unrounded P), o = O / l, LSE = m + ln l.
 * Arguments, direct rows and errors as snapmla_decode (without kv_scale); the
 * other rows are complete after snapmla_combine with the same split plan.
 */
int snapmla_decode_bf16(const void* q_nope, const void* q_rope, const void* kv_latent, const void* k_rope,
                        const int32_t* page_table, const int32_t* seq_lens,
                        int32_t B, int32_t q_len, int32_t H,
                        int32_t max_pages, int32_t num_pages, int32_t page_size,
                        float softmax_scale, int32_t causal,
                        int32_t num_splits, int32_t kv_chunk_tokens,
                        void* workspace, size_t workspace_bytes,
                        void* out, int32_t out_dtype, float* lse,
                        hipStream_t stream);

/*
 * snapmla_append_bf16 -- the step's new tokens into a BF16 cache (the
 * counterpart of snapmla_quantize_append for snapmla_decode_bf16): token t of
 * sequence b goes to position seq_lens[b] - n_new + t, its latent and RoPE rows
 * copied bit for bit.  Arguments and skipped tokens as snapmla_quantize_append.
 */
int snapmla_append_bf16(const void* c_kv_new, const void* k_rope_new, const int32_t* page_table,
                        const int32_t* seq_lens, int32_t B, int32_t n_new, int32_t max_pages, int32_t num_pages,
                        int32_t page_size, void* kv_latent, void* k_rope, hipStream_t stream);

/*
 * snapmla_combine -- split-KV log-sum-exp merge of the partial results that
 * snapmla_decode left in `workspace` (same B, q_len, H, num_splits,
 * kv_chunk_tokens and seq_lens as that call).  Per row:
 *     LSE = log sum_i exp(LSE_i),  o = sum_i exp(LSE_i - LSE) o_i
 * over the row's non-empty pieces.  A row that sees no token gets o = 0 and
 * LSE = -inf; a sequence flagged by a data error gets NaN.  When the decode was
 * given out, the rows it wrote (sequences that at most one piece covers) are
 * left untouched: pass it the same out, out_dtype and lse.
 *
 *   out        [B][q_len][H][512], bf16 (out_dtype 0, round to nearest even) or float32 (1)
 *   lse        float32 [B][q_len][H], natural log of the sum of exp(s) (may be NULL)
 */
int snapmla_combine(const void* workspace, size_t workspace_bytes, const int32_t* seq_lens,
                    int32_t B, int32_t q_len, int32_t H,
                    int32_t num_splits, int32_t kv_chunk_tokens,
                    void* out, int32_t out_dtype, float* lse,
                    hipStream_t stream);

/*
 * snapmla_fetch_dequant -- fused fetch-and-dequantize of the paged cache into
 * BF16 rows (Section 3.3, Fused-Fetch-Dequant: for phases that reuse the cache
 * at high precision, such as chunk prefill or prefix caching; the FP8 rows are
 * dequantized in registers right after the load, in one pass).
 *
 * Sequence b has cu_seqlens[b+1] - cu_seqlens[b] cached tokens (its tokens
 * 0, 1, ...); token j is written to output row cu_seqlens[b] + j:
 *     out[row][0:512]   = bf16( fp32( E4M3(code_i) * sigma_K ) )   (round to nearest even)
 *     out[row][512:576] = the token's RoPE key, bit for bit
 * Every token whose page id is outside [0, num_pages), and every token of a
 * sequence longer than max_pages * 64, gets a row of bf16 NaN (0x7FC0).
 * Sequences with cu_seqlens[b+1] <= cu_seqlens[b] write nothing.
 *
 *   kv_latent, kv_scale, k_rope, page_table   cache (layout above), device, read
 *   cu_seqlens  int32 [B+1]        device, read: output row offsets (nondecreasing)
 *   out         bf16 [cu_seqlens[B]][576]   device, written (the caller sizes it
 *                                            from cu_seqlens[B]; only those rows are written)
 *   0 <= B <= 65535, max_pages >= 1, num_pages >= 1, page_size == 64
 */
int snapmla_fetch_dequant(const uint8_t* kv_latent, const float* kv_scale, const void* k_rope,
                          const int32_t* page_table, const int32_t* cu_seqlens,
                          int32_t B, int32_t max_pages, int32_t num_pages, int32_t page_size,
                          void* out, hipStream_t stream);

/*
 * snapmla_quantize_cache_config -- the KV-cache quantizers of the accuracy
 * ablation (Appendix G, Table 3), for measuring the decode's error under each
 * granularity.  Writes the same cache planes as snapmla_quantize_append for a
 * whole batch: token j of sequence b (cu_seqlens[b+1] - cu_seqlens[b] tokens) is
 * input row cu_seqlens[b] + j and goes to page page_table[b][j / 64], slot j % 64.
 * Every scale is max(fp32(amax / 448), 2^-40) over the configuration's group and
 * every code E4M3_rne(fp32(x / sigma)) (IEEE float32 divisions):
 *   config 0  per-token content, RoPE copied (the method; = quantize_append)
 *   config 1  per-token over the 576 values of content and RoPE together; the RoPE
 *             row stored as bf16(fp32(sigma * E4M3(r / sigma)))  (RoPE-unaware)
 *   config 2  per-tensor static: sigma = 1 (values beyond 448 saturate)
 *   config 3  per-tensor dynamic: one sigma from the amax of all content values
 *   config 4  per-block: one sigma per 64-token page of a sequence
 * Tokens past max_pages * 64 or on a page id outside [0, num_pages) are skipped.
 *
 *   c_kv     bf16 [cu_seqlens[B]][512], k_rope bf16 [cu_seqlens[B]][64]   device, read
 *   page_table int32 [B][max_pages], cu_seqlens int32 [B+1]               device, read
 *   scratch  device uint32 word used by config 3 (may be NULL otherwise); calls that
 *            share it must not overlap
 *   kv_latent, kv_scale, k_rope_out   cache planes, written at the batch's slots
 *   0 <= config <= 4, 0 <= B <= 65535, max_pages >= 1, num_pages >= 1, page_size == 64
 */
int snapmla_quantize_cache_config(const void* c_kv, const void* k_rope, const int32_t* page_table,
                                  const int32_t* cu_seqlens, int32_t B, int32_t max_pages, int32_t num_pages,
                                  int32_t page_size, int32_t config, uint32_t* scratch, uint8_t* kv_latent,
                                  float* kv_scale, void* k_rope_out, hipStream_t stream);

/*
 * snapmla_e4m3_encode -- test hook: E4M3 codes of n float32 values through the
 * same device conversion the quantizers use (round to nearest even, values at
 * or beyond 464 in magnitude saturate to +-448).  x, codes: device; n >= 0.
 */
int snapmla_e4m3_encode(const float* x, int64_t n, uint8_t* codes, hipStream_t stream);

/*
 * snapmla_debug_read_ceiling -- measurement hook, not part of the attention
 * path: streams the cache pages of nblk 64-token blocks into LDS with the same
 * direct-to-LDS copy structure and ring depth as snapmla_decode (latent three
 * blocks ahead, RoPE and scales two), without any attention arithmetic.  Its
 * duration is the read-stream ceiling of that page stream, against which the
 * decode's bandwidth is reported.
 *   kv_latent, kv_scale, k_rope   cache planes (device, read; 16-byte aligned)
 *   pages   int32 [nblk]  physical page of each block in stream order (device,
 *           read); ids outside [0, num_pages) read page 0
 *   units   workgroups; unit u streams blocks [u*nblk/units, (u+1)*nblk/units),
 *           at most 1792 of them (SNAPMLA_INVALID_ARGUMENT otherwise)
 *   out     uint32 [units] (device, written): per unit, the XOR over its blocks
 *           of the first 256 dwords of the latent page and of the RoPE page
 *           (each dword XORed with its counterpart), folded over the 256
 *           dword positions, so a test can check that every page was read
 */
int snapmla_debug_read_ceiling(const uint8_t* kv_latent, const float* kv_scale, const void* k_rope,
                               const int32_t* pages, int32_t nblk, int32_t num_pages, int32_t units,
                               uint32_t* out, hipStream_t stream);

/*
 * snapmla_debug_read_stream -- measurement only: `bytes` of device memory read
 * once by the simplest streaming kernel (16-byte vector loads, grid-stride loop,
 * consecutive lanes on consecutive words, `grid` workgroups of 256 threads).
 * Its duration is the plain read-stream rate of the memory system, the second
 * reference figure (beside the 8 TB/s peak) for the decode's bandwidth.
 *   buf    device, read; 16-byte aligned; bytes a multiple of 16, >= 0
 *   grid   1 .. 2^20 workgroups
 *   out    uint32 [grid] (device, written): per workgroup, the XOR of every
 *          dword it read (workgroup g reads the 16-byte words i with
 *          (i / 256) % grid == g), so a test can check the reads
 */
int snapmla_debug_read_stream(const void* buf, int64_t bytes, int32_t grid, uint32_t* out, hipStream_t stream);

/*
 * snapmla_debug_decode_kernel -- measurement only: the decode launch of
 * snapmla_decode (Algorithm 1 over the KV pieces) without its preparation launch,
 * so that events around it time the decode kernel alone.  The workspace must hold
 * what a snapmla_decode (or snapmla_append_decode) call with the same arguments,
 * on the same stream, prepared: the quantized queries, the split plan and the
 * start descriptors; the call then writes the same partials, direct rows and
 * log-sum-exps as that call's decode launch.  Arguments, layouts, validation and
 * status codes as snapmla_decode; in addition, SNAPMLA_INVALID_ARGUMENT when the
 * last preparation written into this workspace was not an FP8 decode call with the
 * same q_nope and seq_lens buffers, B, q_len, H, num_splits and kv_chunk_tokens
 * (the library records each preparation launch per workspace; the buffers'
 * contents and the stream order are not checked).
 */
int snapmla_debug_decode_kernel(const void* q_nope, const void* q_rope, const uint8_t* kv_latent,
                                const float* kv_scale, const void* k_rope, const int32_t* page_table,
                                const int32_t* seq_lens, int32_t B, int32_t q_len, int32_t H,
                                int32_t max_pages, int32_t num_pages, int32_t page_size,
                                float softmax_scale, int32_t causal, int32_t num_splits,
                                int32_t kv_chunk_tokens, int32_t flags, void* workspace,
                                size_t workspace_bytes, void* out, int32_t out_dtype, float* lse,
                                hipStream_t stream);

/*
 * snapmla_debug_mfma_fp8 -- test hook: the FP8 matrix-core dot product the decode's
 * QK content term is formed with (Section 3.1 runs that GEMM on FP8 matrix
 * cores).  For every tile t, one 16x16x128 FP8 MFMA from a zero accumulator:
 *     c[t][m][n] = sum_k E4M3(a[t][m][k]) * E4M3(b[t][n][k])
 * as the instruction forms it (groups of eight consecutive k, each product
 * truncated below the group's largest exponent sum, the group sums added in
 * float32), so a test can compare the instruction with the oracle's model.
 *   a, b   uint8 [tiles][16][128] E4M3 codes (device, read; 16-byte aligned)
 *   c      float [tiles][16][16] (device, written)
 *   0 <= tiles <= 2^31 - 1
 */
int snapmla_debug_mfma_fp8(const uint8_t* a, const uint8_t* b, float* c, int64_t tiles, hipStream_t stream);

/*
 * snapmla_debug_set_spin_limit -- test hook: the bound on the polls of every
 * handshake wait inside the decode kernels of later snapmla_decode,
 * snapmla_append_decode and snapmla_decode_bf16 calls of this process (default
 * 4194304).  The waits end by construction; the bound only guarantees that a
 * kernel terminates.  A wait that reaches it marks its KV piece, whose outputs
 * and LSEs then come out NaN, so a lost handshake is visible rather than
 * silently stale.  With polls = 0 every wait gives up after its first poll (every output
 * NaN), which lets a test check that path without hanging anything.
 *   polls >= 0 (SNAPMLA_INVALID_ARGUMENT otherwise).  Process-wide; not for
 *   concurrent use with decode calls on other threads.
 */
int snapmla_debug_set_spin_limit(int32_t polls);

#ifdef __cplusplus
}
#endif

#endif /* SNAPMLA_H */
