// C ABI of libsnapmla.so (declared in include/snapmla.h): argument validation,
// workspace carve-up and kernel launches on the caller's stream.

#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>
#include <unordered_map>

#include "snapmla.h"
#include "snapmla_internal.h"

namespace {

thread_local std::string g_last_error;
std::atomic<int> g_spin_limit{snapmla::kDefaultSpinLimit};

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int ok() {
  g_last_error.clear();
  return SNAPMLA_OK;
}

bool misaligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }
bool misaligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) != 0; }

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

int hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(SNAPMLA_HIP_ERROR, "%s: %s", what, hipGetErrorString(e));
}

int check_shapes(int32_t B, int32_t q_len, int32_t H, int32_t num_splits, int32_t kv_chunk_tokens) {
  if (B < 0) return fail(SNAPMLA_INVALID_ARGUMENT, "B must be >= 0 (got %d)", B);
  if (q_len != 1 && q_len != 2) return fail(SNAPMLA_INVALID_ARGUMENT, "q_len must be 1 or 2 (got %d)", q_len);
  if (H < 1) return fail(SNAPMLA_INVALID_ARGUMENT, "H must be >= 1 (got %d)", H);
  if ((int64_t)q_len * H > 256)
    return fail(SNAPMLA_INVALID_ARGUMENT, "q_len*H must be <= 256 (got %d)", q_len * H);
  if (num_splits < 1) return fail(SNAPMLA_INVALID_ARGUMENT, "num_splits must be >= 1 (got %d)", num_splits);
  if (kv_chunk_tokens > 0 && (int64_t)B * num_splits > (int64_t)1 << 26)
    return fail(SNAPMLA_INVALID_ARGUMENT, "B * num_splits must be <= 2^26 with fixed KV chunks (got %lld)",
                (long long)B * num_splits);
  if (num_splits > (1 << 26)) return fail(SNAPMLA_INVALID_ARGUMENT, "num_splits must be <= 2^26 (got %d)", num_splits);
  if (kv_chunk_tokens < 0 || kv_chunk_tokens % 64 != 0)
    return fail(SNAPMLA_INVALID_ARGUMENT, "kv_chunk_tokens must be 0 or a positive multiple of 64 (got %d)",
                kv_chunk_tokens);
  return SNAPMLA_OK;
}

// snapmla_decode and snapmla_decode_bf16: validation, workspace carve-up, the prep
// launch (query quantization only for the FP8 cache) and the decode launch.
// New tokens that snapmla_append_decode quantizes and appends inside the decode's
// preparation launch (n_new == 0: none).
struct AppendIn {
  const void* c_kv_new = nullptr;
  const void* k_rope_new = nullptr;
  int32_t n_new = 0;
};

// What the last FP8 preparation launch into each workspace was made from.  The decode
// launch alone (snapmla_debug_decode_kernel) reads the start descriptors, block prefix
// and quantized queries that launch wrote; with a workspace no matching call prepared
// those words are undefined and the kernel could address pages out of bounds, so the
// entry point refuses it on the host.  (Only the buffers and sizes are compared: keeping
// the contents of seq_lens and q_nope unchanged, and ordering the launch after the
// preparation, stay the caller's part.)
struct PrepKey {
  const void* q_nope = nullptr;
  const int32_t* seq_lens = nullptr;
  int32_t B = 0, q_len = 0, H = 0, num_splits = 0, kv_chunk_tokens = 0;
  bool operator==(const PrepKey& o) const {
    return q_nope == o.q_nope && seq_lens == o.seq_lens && B == o.B && q_len == o.q_len &&
           H == o.H && num_splits == o.num_splits && kv_chunk_tokens == o.kv_chunk_tokens;
  }
};
std::mutex g_prep_mu;
std::unordered_map<const void*, PrepKey> g_prepared;   // workspace -> its last FP8 preparation
constexpr size_t kMaxPreparedRecords = 4096;           // bounded: cleared when full

int decode_common(const void* q_nope, const void* q_rope, const void* kv_latent, const float* kv_scale,
                  const void* k_rope, const int32_t* page_table, const int32_t* seq_lens, int32_t B,
                  int32_t q_len, int32_t H, int32_t max_pages, int32_t num_pages, int32_t page_size,
                  float softmax_scale, int32_t causal, int32_t num_splits, int32_t kv_chunk_tokens,
                  void* workspace, size_t workspace_bytes, void* out, int32_t out_dtype, float* lse,
                  hipStream_t stream, bool bf16_cache, const AppendIn& app = AppendIn(), int32_t flags = 0,
                  bool run_prep = true) {
  int st = check_shapes(B, q_len, H, num_splits, kv_chunk_tokens);
  if (st != SNAPMLA_OK) return st;
  if ((flags & ~SNAPMLA_DECODE_EXACT_QK) != 0)
    return fail(SNAPMLA_INVALID_ARGUMENT, "unknown decode flags 0x%x", (unsigned)flags);
  if (out_dtype != 0 && out_dtype != 1) return fail(SNAPMLA_INVALID_ARGUMENT, "out_dtype must be 0 or 1");
  if (!out && lse) return fail(SNAPMLA_INVALID_ARGUMENT, "lse without out: pass both or neither");
  if (page_size != 64) return fail(SNAPMLA_UNSUPPORTED, "page_size must be 64 (got %d)", page_size);
  if (max_pages < 1 || num_pages < 1)
    return fail(SNAPMLA_INVALID_ARGUMENT, "max_pages and num_pages must be >= 1 (got %d, %d)", max_pages, num_pages);
  if (!(softmax_scale > 0.0f) || !std::isfinite(softmax_scale))
    return fail(SNAPMLA_INVALID_ARGUMENT, "softmax_scale must be finite and > 0");
  if (causal != 0 && causal != 1) return fail(SNAPMLA_INVALID_ARGUMENT, "causal must be 0 or 1");
  if ((int64_t)max_pages * 64 > 0x7FFFFFFF) return fail(SNAPMLA_INVALID_ARGUMENT, "max_pages too large");
  const snapmla::WsLayout L = snapmla::ws_layout(B, q_len, H, num_splits, kv_chunk_tokens);
  if (B == 0) return ok();
  // Direct rows (out/lse written by the decode for sequences that one piece covers): the
  // FP8-cache kernel writes them with one row group (R <= 64); with several it writes
  // partials only and the combine writes every row.  The BF16-cache kernel writes them
  // for any R.
  void* dout = (bf16_cache || L.G == 1) ? out : nullptr;
  float* dlse = dout ? lse : nullptr;
  if (!q_nope || !q_rope || !kv_latent || (!bf16_cache && !kv_scale) || !k_rope || !page_table || !seq_lens ||
      !workspace)
    return fail(SNAPMLA_INVALID_ARGUMENT, "null pointer argument");
  if (misaligned(q_nope) || misaligned(q_rope) || misaligned(kv_latent) || (!bf16_cache && misaligned(kv_scale)) ||
      misaligned(k_rope) || misaligned4(page_table) || misaligned4(seq_lens) || misaligned(workspace) ||
      (out && misaligned(out)) || (lse && misaligned4(lse)))
    return fail(SNAPMLA_MISALIGNED, "pointer misaligned (int32/float32 index arrays need 4 bytes, data buffers 16)");
  if (workspace_bytes < L.total)
    return fail(SNAPMLA_WORKSPACE_TOO_SMALL, "workspace needs %zu bytes (got %zu)", L.total, workspace_bytes);
  const int64_t app_toks = (int64_t)B * app.n_new;
  if (app_toks > 0) {
    if (!app.c_kv_new || !app.k_rope_new) return fail(SNAPMLA_INVALID_ARGUMENT, "null pointer argument");
    if (misaligned(app.c_kv_new) || misaligned(app.k_rope_new))
      return fail(SNAPMLA_MISALIGNED, "c_kv_new and k_rope_new must be 16-byte aligned");
    if ((app_toks + 3) / 4 > 0x3FFFFFFF) return fail(SNAPMLA_INVALID_ARGUMENT, "too many new tokens");
  }

  uint8_t* ws = static_cast<uint8_t*>(workspace);
  snapmla::PrepArgs p;
  p.q_nope = static_cast<const uint16_t*>(q_nope);
  p.q8 = ws + L.q8;
  p.sq = reinterpret_cast<float*>(ws + L.sq);
  // row waves: query quantization (FP8 cache; the BF16 cache reads the bf16 queries as
  // they are) and the rows of sequences without blocks (when out is given)
  p.rows = (!bf16_cache || dout) ? (int64_t)B * L.R : 0;
  p.quantize = !bf16_cache;
  p.ctrl = reinterpret_cast<int32_t*>(ws + L.ctrl);
  p.out = dout;
  p.out_lse = dlse;
  p.out_dtype = out_dtype;
  p.R = L.R;
  p.seq_lens = seq_lens;
  p.prefix = reinterpret_cast<int32_t*>(ws + L.prefix);
  p.flags = reinterpret_cast<int32_t*>(ws + L.flags);
  p.zero = ws + L.zero;
  p.desc = reinterpret_cast<int32_t*>(ws + L.desc);
  p.units = L.units;
  p.pad = L.pad;
  p.B = B;
  p.q_len = q_len;
  p.max_pages = max_pages;
  p.chunk_blocks = kv_chunk_tokens / 64;
  p.num_splits = num_splits;
  if (app_toks > 0) {
    p.c_kv_new = static_cast<const uint16_t*>(app.c_kv_new);
    p.k_rope_new = static_cast<const uint16_t*>(app.k_rope_new);
    p.page_table = page_table;
    p.kv_latent = static_cast<uint8_t*>(const_cast<void*>(kv_latent));
    p.kv_scale = const_cast<float*>(kv_scale);
    p.k_rope = static_cast<uint16_t*>(const_cast<void*>(k_rope));
    p.n_new = app.n_new;
    p.num_pages = num_pages;
    p.ablocks = (int)((app_toks + 3) / 4);
  }
  PrepKey key;
  key.q_nope = q_nope;
  key.seq_lens = seq_lens;
  key.B = B;
  key.q_len = q_len;
  key.H = H;
  key.num_splits = num_splits;
  key.kv_chunk_tokens = kv_chunk_tokens;
  if (run_prep) {
    hipError_t e = snapmla::launch_prep(p, stream);
    if (e != hipSuccess) return hip_status(e, "decode prep launch");
    std::lock_guard<std::mutex> lk(g_prep_mu);
    if (bf16_cache) {
      g_prepared.erase(workspace);
    } else {
      if (g_prepared.size() >= kMaxPreparedRecords) g_prepared.clear();
      g_prepared[workspace] = key;
    }
  } else {
    std::lock_guard<std::mutex> lk(g_prep_mu);
    auto it = g_prepared.find(workspace);
    if (bf16_cache || it == g_prepared.end() || !(it->second == key))
      return fail(SNAPMLA_INVALID_ARGUMENT,
                  "workspace not prepared by an FP8 decode call with these queries, lengths and sizes");
  }

  snapmla::DecodeArgs d;
  d.q_nope = static_cast<const uint16_t*>(q_nope);
  d.q8 = p.q8;
  d.sq = p.sq;
  d.q_rope = static_cast<const uint16_t*>(q_rope);
  d.kv_latent = static_cast<const uint8_t*>(kv_latent);
  d.kv_scale = kv_scale;
  d.k_rope = static_cast<const uint16_t*>(k_rope);
  d.page_table = page_table;
  d.seq_lens = seq_lens;
  d.prefix = p.prefix;
  d.desc = p.desc;
  d.zero = p.zero;
  d.part_o = reinterpret_cast<float*>(ws + L.o);
  d.part_lse = reinterpret_cast<float*>(ws + L.lse);
  d.B = B;
  d.q_len = q_len;
  d.H = H;
  d.R = L.R;
  d.G = L.G;
  d.rows_pad = L.rows_pad;
  d.max_pages = max_pages;
  d.num_pages = num_pages;
  d.causal = causal;
  d.num_splits = num_splits;
  d.chunk_blocks = kv_chunk_tokens / 64;
  d.sl2 = softmax_scale * 1.4426950408889634f;
  d.spin_limit = snapmla::spin_limit();
  d.qk_exact = (flags & SNAPMLA_DECODE_EXACT_QK) != 0 ? 1 : 0;
  d.out = dout;
  d.out_lse = dlse;
  d.out_dtype = out_dtype;
  if (bf16_cache)
    return hip_status(snapmla::launch_decode_bf16(d, static_cast<const uint16_t*>(kv_latent), stream),
                      "decode_bf16 launch");
  return hip_status(snapmla::launch_decode(d, stream), "decode launch");
}

}  // namespace

namespace snapmla {

int spin_limit() { return g_spin_limit.load(std::memory_order_relaxed); }

WsLayout ws_layout(int B, int q_len, int H, int num_splits, int kv_chunk_tokens) {
  WsLayout L;
  L.R = q_len * H;
  L.G = (L.R + 63) / 64;
  L.rows_pad = 64 * L.G;
  L.pieces = kv_chunk_tokens == 0 ? num_splits + B : B * num_splits;
  const size_t rows = (size_t)B * L.R;
  size_t off = 0;
  L.q8 = off;     off += align256(rows * 512);
  L.sq = off;     off += align256(rows * 4);
  L.prefix = off; off += align256(((size_t)B + 1) * 4);
  L.flags = off;  off += align256((size_t)B * 4);
  L.zero = off;   off += 1024;
  L.ctrl = off;   off += 256;
  L.units = kv_chunk_tokens == 0 ? num_splits : B * num_splits;   // <= 2^26 (check_shapes)
  L.pad = kv_chunk_tokens == 0 && L.G == 1 ? kPlanPad : 0;
  L.desc = off;   off += align256((size_t)L.units * kDescInts * 4);
  L.lse = off;    off += align256((size_t)L.pieces * L.rows_pad * 4);
  L.o = off;      off += align256((size_t)L.pieces * L.rows_pad * 512 * 4);
  L.total = off;
  return L;
}

}  // namespace snapmla

extern "C" {

int snapmla_abi_version(void) { return SNAPMLA_ABI_VERSION; }

const char* snapmla_get_last_error(void) { return g_last_error.c_str(); }

int snapmla_debug_mfma_fp8(const uint8_t* a, const uint8_t* b, float* c, int64_t tiles, hipStream_t stream) {
  if (tiles < 0 || tiles > 0x7FFFFFFF) return fail(SNAPMLA_INVALID_ARGUMENT, "tiles out of range (got %lld)",
                                                   (long long)tiles);
  if (tiles == 0) return ok();
  if (!a || !b || !c) return fail(SNAPMLA_INVALID_ARGUMENT, "null pointer argument");
  if (misaligned(a) || misaligned(b) || misaligned(c)) return fail(SNAPMLA_MISALIGNED, "pointers must be 16-byte aligned");
  return hip_status(snapmla::launch_mfma_fp8(a, b, c, tiles, stream), "mfma_fp8 launch");
}

int snapmla_debug_set_spin_limit(int32_t polls) {
  if (polls < 0) return fail(SNAPMLA_INVALID_ARGUMENT, "polls must be >= 0 (got %d)", polls);
  g_spin_limit.store(polls == 0 ? 0 : polls, std::memory_order_relaxed);
  return ok();
}

int snapmla_quantize_append(const void* c_kv_new, const void* k_rope_new, const int32_t* page_table,
                            const int32_t* seq_lens, int32_t B, int32_t n_new, int32_t max_pages,
                            int32_t num_pages, int32_t page_size, uint8_t* kv_latent, float* kv_scale,
                            void* k_rope, hipStream_t stream) {
  if (page_size != 64) return fail(SNAPMLA_UNSUPPORTED, "page_size must be 64 (got %d)", page_size);
  if (B < 0 || n_new < 0) return fail(SNAPMLA_INVALID_ARGUMENT, "B and n_new must be >= 0 (got %d, %d)", B, n_new);
  if (max_pages < 1 || num_pages < 1)
    return fail(SNAPMLA_INVALID_ARGUMENT, "max_pages and num_pages must be >= 1 (got %d, %d)", max_pages, num_pages);
  if ((int64_t)B * n_new == 0) return ok();
  if (!c_kv_new || !k_rope_new || !page_table || !seq_lens || !kv_latent || !kv_scale || !k_rope)
    return fail(SNAPMLA_INVALID_ARGUMENT, "null pointer argument");
  if (misaligned(c_kv_new) || misaligned(k_rope_new) || misaligned4(page_table) || misaligned4(seq_lens) ||
      misaligned(kv_latent) || misaligned(kv_scale) || misaligned(k_rope))
    return fail(SNAPMLA_MISALIGNED, "pointer misaligned (int32/float32 index arrays need 4 bytes, data buffers 16)");
  return hip_status(snapmla::launch_append(static_cast<const uint16_t*>(c_kv_new),
                                           static_cast<const uint16_t*>(k_rope_new), page_table, seq_lens, B,
                                           n_new, max_pages, num_pages, kv_latent, kv_scale,
                                           static_cast<uint16_t*>(k_rope), stream),
                    "quantize_append launch");
}

int snapmla_quantize_rows(const void* x, int64_t rows, uint8_t* codes, float* scale, hipStream_t stream) {
  if (rows < 0) return fail(SNAPMLA_INVALID_ARGUMENT, "rows must be >= 0 (got %lld)", (long long)rows);
  if (rows == 0) return ok();
  if (!x || !codes || !scale) return fail(SNAPMLA_INVALID_ARGUMENT, "null pointer argument");
  if (misaligned(x) || misaligned(codes) || misaligned(scale))
    return fail(SNAPMLA_MISALIGNED, "pointer misaligned (int32/float32 index arrays need 4 bytes, data buffers 16)");
  return hip_status(snapmla::launch_quantize_rows(static_cast<const uint16_t*>(x), rows, codes, scale, stream),
                    "quantize_rows launch");
}

int snapmla_e4m3_encode(const float* x, int64_t n, uint8_t* codes, hipStream_t stream) {
  if (n < 0) return fail(SNAPMLA_INVALID_ARGUMENT, "n must be >= 0");
  if (n == 0) return ok();
  if (!x || !codes) return fail(SNAPMLA_INVALID_ARGUMENT, "null pointer argument");
  if (misaligned(x) || misaligned(codes)) return fail(SNAPMLA_MISALIGNED, "pointer misaligned (int32/float32 index arrays need 4 bytes, data buffers 16)");
  return hip_status(snapmla::launch_encode(x, n, codes, stream), "e4m3_encode launch");
}

int snapmla_decode_workspace_size(int32_t B, int32_t q_len, int32_t H, int32_t num_splits,
                                  int32_t kv_chunk_tokens, size_t* bytes) {
  const int st = check_shapes(B, q_len, H, num_splits, kv_chunk_tokens);
  if (st != SNAPMLA_OK) return st;
  if (!bytes) return fail(SNAPMLA_INVALID_ARGUMENT, "bytes must not be null");
  *bytes = snapmla::ws_layout(B, q_len, H, num_splits, kv_chunk_tokens).total;
  return ok();
}

int snapmla_decode(const void* q_nope, const void* q_rope, const uint8_t* kv_latent, const float* kv_scale,
                   const void* k_rope, const int32_t* page_table, const int32_t* seq_lens, int32_t B,
                   int32_t q_len, int32_t H, int32_t max_pages, int32_t num_pages, int32_t page_size,
                   float softmax_scale, int32_t causal, int32_t num_splits, int32_t kv_chunk_tokens,
                   int32_t flags, void* workspace, size_t workspace_bytes, void* out, int32_t out_dtype, float* lse,
                   hipStream_t stream) {
  return decode_common(q_nope, q_rope, kv_latent, kv_scale, k_rope, page_table, seq_lens, B, q_len, H, max_pages,
                       num_pages, page_size, softmax_scale, causal, num_splits, kv_chunk_tokens, workspace,
                       workspace_bytes, out, out_dtype, lse, stream, false, AppendIn(), flags);
}

int snapmla_debug_decode_kernel(const void* q_nope, const void* q_rope, const uint8_t* kv_latent, const float* kv_scale,
                                const void* k_rope, const int32_t* page_table, const int32_t* seq_lens, int32_t B,
                                int32_t q_len, int32_t H, int32_t max_pages, int32_t num_pages, int32_t page_size,
                                float softmax_scale, int32_t causal, int32_t num_splits, int32_t kv_chunk_tokens,
                                int32_t flags, void* workspace, size_t workspace_bytes, void* out, int32_t out_dtype,
                                float* lse, hipStream_t stream) {
  return decode_common(q_nope, q_rope, kv_latent, kv_scale, k_rope, page_table, seq_lens, B, q_len, H, max_pages,
                       num_pages, page_size, softmax_scale, causal, num_splits, kv_chunk_tokens, workspace,
                       workspace_bytes, out, out_dtype, lse, stream, false, AppendIn(), flags, false);
}

int snapmla_append_decode(const void* c_kv_new, const void* k_rope_new, int32_t n_new, const void* q_nope,
                          const void* q_rope, uint8_t* kv_latent, float* kv_scale, void* k_rope,
                          const int32_t* page_table, const int32_t* seq_lens, int32_t B, int32_t q_len, int32_t H,
                          int32_t max_pages, int32_t num_pages, int32_t page_size, float softmax_scale,
                          int32_t causal, int32_t num_splits, int32_t kv_chunk_tokens, int32_t flags,
                          void* workspace, size_t workspace_bytes, void* out, int32_t out_dtype, float* lse,
                          hipStream_t stream) {
  if (n_new < 0) return fail(SNAPMLA_INVALID_ARGUMENT, "n_new must be >= 0 (got %d)", n_new);
  AppendIn app;
  app.c_kv_new = c_kv_new;
  app.k_rope_new = k_rope_new;
  app.n_new = n_new;
  return decode_common(q_nope, q_rope, kv_latent, kv_scale, k_rope, page_table, seq_lens, B, q_len, H, max_pages,
                       num_pages, page_size, softmax_scale, causal, num_splits, kv_chunk_tokens, workspace,
                       workspace_bytes, out, out_dtype, lse, stream, false, app, flags);
}

int snapmla_decode_bf16(const void* q_nope, const void* q_rope, const void* kv_latent, const void* k_rope,
                        const int32_t* page_table, const int32_t* seq_lens, int32_t B, int32_t q_len, int32_t H,
                        int32_t max_pages, int32_t num_pages, int32_t page_size, float softmax_scale,
                        int32_t causal, int32_t num_splits, int32_t kv_chunk_tokens, void* workspace,
                        size_t workspace_bytes, void* out, int32_t out_dtype, float* lse, hipStream_t stream) {
  return decode_common(q_nope, q_rope, kv_latent, nullptr, k_rope, page_table, seq_lens, B, q_len, H, max_pages,
                       num_pages, page_size, softmax_scale, causal, num_splits, kv_chunk_tokens, workspace,
                       workspace_bytes, out, out_dtype, lse, stream, true);
}

int snapmla_append_bf16(const void* c_kv_new, const void* k_rope_new, const int32_t* page_table,
                        const int32_t* seq_lens, int32_t B, int32_t n_new, int32_t max_pages, int32_t num_pages,
                        int32_t page_size, void* kv_latent, void* k_rope, hipStream_t stream) {
  if (page_size != 64) return fail(SNAPMLA_UNSUPPORTED, "page_size must be 64 (got %d)", page_size);
  if (B < 0 || n_new < 0) return fail(SNAPMLA_INVALID_ARGUMENT, "B and n_new must be >= 0 (got %d, %d)", B, n_new);
  if (max_pages < 1 || num_pages < 1)
    return fail(SNAPMLA_INVALID_ARGUMENT, "max_pages and num_pages must be >= 1 (got %d, %d)", max_pages, num_pages);
  if ((int64_t)B * n_new == 0) return ok();
  if (!c_kv_new || !k_rope_new || !page_table || !seq_lens || !kv_latent || !k_rope)
    return fail(SNAPMLA_INVALID_ARGUMENT, "null pointer argument");
  if (misaligned(c_kv_new) || misaligned(k_rope_new) || misaligned(kv_latent) || misaligned(k_rope) ||
      misaligned4(page_table) || misaligned4(seq_lens))
    return fail(SNAPMLA_MISALIGNED, "pointer misaligned (int32 index arrays need 4 bytes, data buffers 16)");
  return hip_status(snapmla::launch_append_bf16(static_cast<const uint16_t*>(c_kv_new),
                                                static_cast<const uint16_t*>(k_rope_new), page_table, seq_lens, B,
                                                n_new, max_pages, num_pages, static_cast<uint16_t*>(kv_latent),
                                                static_cast<uint16_t*>(k_rope), stream),
                    "append_bf16 launch");
}

int snapmla_combine(const void* workspace, size_t workspace_bytes, const int32_t* seq_lens, int32_t B,
                    int32_t q_len, int32_t H, int32_t num_splits, int32_t kv_chunk_tokens, void* out,
                    int32_t out_dtype, float* lse, hipStream_t stream) {
  int st = check_shapes(B, q_len, H, num_splits, kv_chunk_tokens);
  if (st != SNAPMLA_OK) return st;
  if (out_dtype != 0 && out_dtype != 1) return fail(SNAPMLA_INVALID_ARGUMENT, "out_dtype must be 0 or 1");
  const snapmla::WsLayout L = snapmla::ws_layout(B, q_len, H, num_splits, kv_chunk_tokens);
  if (B == 0) return ok();
  if (!workspace || !seq_lens || !out) return fail(SNAPMLA_INVALID_ARGUMENT, "null pointer argument");
  if (misaligned(workspace) || misaligned4(seq_lens) || misaligned(out) || (lse && misaligned4(lse)))
    return fail(SNAPMLA_MISALIGNED, "pointer misaligned (int32/float32 index arrays need 4 bytes, data buffers 16)");
  if (workspace_bytes < L.total)
    return fail(SNAPMLA_WORKSPACE_TOO_SMALL, "workspace needs %zu bytes (got %zu)", L.total, workspace_bytes);
  const uint8_t* ws = static_cast<const uint8_t*>(workspace);
  snapmla::CombineArgs c;
  c.part_o = reinterpret_cast<const float*>(ws + L.o);
  c.part_lse = reinterpret_cast<const float*>(ws + L.lse);
  c.prefix = reinterpret_cast<const int32_t*>(ws + L.prefix);
  c.flags = reinterpret_cast<const int32_t*>(ws + L.flags);
  c.ctrl = reinterpret_cast<const int32_t*>(ws + L.ctrl);
  c.seq_lens = seq_lens;
  c.out = out;
  c.lse = lse;
  c.B = B;
  c.q_len = q_len;
  c.H = H;
  c.R = L.R;
  c.rows_pad = L.rows_pad;
  c.num_splits = num_splits;
  c.chunk_blocks = kv_chunk_tokens / 64;
  c.out_dtype = out_dtype;
  c.pad = L.pad;
  return hip_status(snapmla::launch_combine(c, stream), "combine launch");
}

int snapmla_fetch_dequant(const uint8_t* kv_latent, const float* kv_scale, const void* k_rope,
                          const int32_t* page_table, const int32_t* cu_seqlens, int32_t B, int32_t max_pages,
                          int32_t num_pages, int32_t page_size, void* out, hipStream_t stream) {
  if (page_size != 64) return fail(SNAPMLA_UNSUPPORTED, "page_size must be 64 (got %d)", page_size);
  if (B < 0 || B > 65535) return fail(SNAPMLA_INVALID_ARGUMENT, "B must be in [0, 65535] (got %d)", B);
  if (max_pages < 1 || num_pages < 1)
    return fail(SNAPMLA_INVALID_ARGUMENT, "max_pages and num_pages must be >= 1 (got %d, %d)", max_pages, num_pages);
  if (B == 0) return ok();
  if (!kv_latent || !kv_scale || !k_rope || !page_table || !cu_seqlens || !out)
    return fail(SNAPMLA_INVALID_ARGUMENT, "null pointer");
  if (misaligned(kv_latent) || misaligned(kv_scale) || misaligned(k_rope) || misaligned(out))
    return fail(SNAPMLA_MISALIGNED, "kv_latent, kv_scale, k_rope and out must be 16-byte aligned");
  if (misaligned4(page_table) || misaligned4(cu_seqlens))
    return fail(SNAPMLA_MISALIGNED, "page_table and cu_seqlens must be 4-byte aligned");
  snapmla::FetchArgs a;
  a.kv_latent = kv_latent;
  a.kv_scale = kv_scale;
  a.k_rope = static_cast<const uint16_t*>(k_rope);
  a.page_table = page_table;
  a.cu = cu_seqlens;
  a.out = static_cast<uint16_t*>(out);
  a.B = B;
  a.max_pages = max_pages;
  a.num_pages = num_pages;
  return hip_status(snapmla::launch_fetch_dequant(a, stream), "fetch_dequant launch");
}

int snapmla_quantize_cache_config(const void* c_kv, const void* k_rope, const int32_t* page_table,
                                  const int32_t* cu_seqlens, int32_t B, int32_t max_pages, int32_t num_pages,
                                  int32_t page_size, int32_t config, uint32_t* scratch, uint8_t* kv_latent,
                                  float* kv_scale, void* k_rope_out, hipStream_t stream) {
  if (page_size != 64) return fail(SNAPMLA_UNSUPPORTED, "page_size must be 64 (got %d)", page_size);
  if (config < 0 || config > 4) return fail(SNAPMLA_INVALID_ARGUMENT, "config must be 0..4 (got %d)", config);
  if (B < 0 || B > 65535) return fail(SNAPMLA_INVALID_ARGUMENT, "B must be in [0, 65535] (got %d)", B);
  if (max_pages < 1 || num_pages < 1)
    return fail(SNAPMLA_INVALID_ARGUMENT, "max_pages and num_pages must be >= 1 (got %d, %d)", max_pages, num_pages);
  if (B == 0) return ok();
  if (!c_kv || !k_rope || !page_table || !cu_seqlens || !kv_latent || !kv_scale || !k_rope_out ||
      (config == 3 && !scratch))
    return fail(SNAPMLA_INVALID_ARGUMENT, "null pointer");
  if (misaligned(c_kv) || misaligned(k_rope) || misaligned(kv_latent) || misaligned(kv_scale) ||
      misaligned(k_rope_out))
    return fail(SNAPMLA_MISALIGNED, "c_kv, k_rope, kv_latent, kv_scale and k_rope_out must be 16-byte aligned");
  if (misaligned4(page_table) || misaligned4(cu_seqlens) || (scratch && misaligned4(scratch)))
    return fail(SNAPMLA_MISALIGNED, "page_table, cu_seqlens and scratch must be 4-byte aligned");
  return hip_status(snapmla::launch_quantize_cache_config(
                        static_cast<const uint16_t*>(c_kv), static_cast<const uint16_t*>(k_rope), page_table,
                        cu_seqlens, B, max_pages, num_pages, config, scratch, kv_latent, kv_scale,
                        static_cast<uint16_t*>(k_rope_out), stream),
                    "quantize_cache_config launch");
}

}  // extern "C"

int snapmla_debug_read_ceiling(const uint8_t* kv_latent, const float* kv_scale, const void* k_rope,
                               const int32_t* pages, int32_t nblk, int32_t num_pages, int32_t units,
                               uint32_t* out, hipStream_t stream) {
  if (nblk < 0) return fail(SNAPMLA_INVALID_ARGUMENT, "nblk must be >= 0 (got %d)", nblk);
  if (units < 1 || units > (1 << 20)) return fail(SNAPMLA_INVALID_ARGUMENT, "units must be in [1, 2^20] (got %d)", units);
  if (num_pages < 1) return fail(SNAPMLA_INVALID_ARGUMENT, "num_pages must be >= 1 (got %d)", num_pages);
  if (((int64_t)nblk + units - 1) / units > snapmla::kCeilingMaxBlocks)
    return fail(SNAPMLA_INVALID_ARGUMENT, "at most %d blocks per unit: use units >= %lld", snapmla::kCeilingMaxBlocks,
                (long long)(((int64_t)nblk + snapmla::kCeilingMaxBlocks - 1) / snapmla::kCeilingMaxBlocks));
  if (!out || (nblk > 0 && (!kv_latent || !kv_scale || !k_rope || !pages)))
    return fail(SNAPMLA_INVALID_ARGUMENT, "null pointer");
  if (misaligned(kv_latent) || misaligned(kv_scale) || misaligned(k_rope))
    return fail(SNAPMLA_MISALIGNED, "kv_latent, kv_scale and k_rope must be 16-byte aligned");
  if (misaligned4(pages) || misaligned4(out)) return fail(SNAPMLA_MISALIGNED, "pages and out must be 4-byte aligned");
  snapmla::CeilingArgs a;
  a.kv_latent = kv_latent;
  a.kv_scale = kv_scale;
  a.k_rope = static_cast<const uint16_t*>(k_rope);
  a.pages = pages;
  a.out = out;
  a.nblk = nblk;
  a.num_pages = num_pages;
  a.units = units;
  return hip_status(snapmla::launch_read_ceiling(a, stream), "read_ceiling launch");
}

int snapmla_debug_read_stream(const void* buf, int64_t bytes, int32_t grid, uint32_t* out, hipStream_t stream) {
  if (bytes < 0 || bytes % 16 != 0)
    return fail(SNAPMLA_INVALID_ARGUMENT, "bytes must be a non-negative multiple of 16 (got %lld)", (long long)bytes);
  if (grid < 1 || grid > (1 << 20)) return fail(SNAPMLA_INVALID_ARGUMENT, "grid must be in [1, 2^20] (got %d)", grid);
  if (!out || (bytes > 0 && !buf)) return fail(SNAPMLA_INVALID_ARGUMENT, "null pointer");
  if (misaligned(buf)) return fail(SNAPMLA_MISALIGNED, "buf must be 16-byte aligned");
  if (misaligned4(out)) return fail(SNAPMLA_MISALIGNED, "out must be 4-byte aligned");
  return hip_status(snapmla::launch_read_stream(buf, bytes / 16, grid, out, stream), "read_stream launch");
}

// ---- the decode step without a caller workspace ------------------------------
// snapmla_append_decode_noalloc keeps its workspace in this file-scope array
// (each GPU the library runs on holds its own copy until the process ends).  In
// host code `scratch` only names the array: its device address on the current
// GPU comes from hipGetSymbolAddress, taken once per device and cached below,
// and only that address is handed to kernels.
static __device__ __align__(256) uint8_t scratch[SNAPMLA_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_addr[kMaxDevices] = {};   // device address of `scratch` per device, null until resolved

int scratch_address(void** addr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(SNAPMLA_UNSUPPORTED, "device %d is beyond the %d devices the scratch table holds", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_addr[dev]) {
    void* a = nullptr;
    e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, "hipGetSymbolAddress(scratch)");
    if (!a) return fail(SNAPMLA_HIP_ERROR, "hipGetSymbolAddress(scratch) gave a null address");
    g_scratch_addr[dev] = a;
  }
  *addr = g_scratch_addr[dev];
  return SNAPMLA_OK;
}

}  // namespace

int snapmla_append_decode_noalloc(const void* c_kv_new, const void* k_rope_new, int32_t n_new, const void* q_nope,
                                  const void* q_rope, uint8_t* kv_latent, float* kv_scale, void* k_rope,
                                  const int32_t* page_table, const int32_t* seq_lens, int32_t B, int32_t q_len,
                                  int32_t H, int32_t max_pages, int32_t num_pages, int32_t page_size,
                                  float softmax_scale, int32_t causal, int32_t num_splits, int32_t kv_chunk_tokens,
                                  int32_t flags, void* out, int32_t out_dtype, float* lse, hipStream_t stream) {
  int st = check_shapes(B, q_len, H, num_splits, kv_chunk_tokens);
  if (st != SNAPMLA_OK) return st;
  const size_t need = snapmla::ws_layout(B, q_len, H, num_splits, kv_chunk_tokens).total;
  if (need > SNAPMLA_NOALLOC_SCRATCH_BYTES)
    return fail(SNAPMLA_WORKSPACE_TOO_SMALL,
                "this call needs %zu bytes of workspace; the static scratch holds %zu (fewer splits or rows per "
                "call, or snapmla_append_decode with a caller workspace)",
                need, (size_t)SNAPMLA_NOALLOC_SCRATCH_BYTES);
  if (out_dtype != 0 && out_dtype != 1) return fail(SNAPMLA_INVALID_ARGUMENT, "out_dtype must be 0 or 1");
  if (n_new < 0) return fail(SNAPMLA_INVALID_ARGUMENT, "n_new must be >= 0 (got %d)", n_new);
  if (B == 0) return ok();
  if (!out) return fail(SNAPMLA_INVALID_ARGUMENT, "null pointer argument");
  if (misaligned(out) || (lse && misaligned4(lse)))
    return fail(SNAPMLA_MISALIGNED, "out must be 16-byte aligned, lse 4-byte aligned");
  void* ws = nullptr;
  st = scratch_address(&ws);
  if (st != SNAPMLA_OK) return st;
  st = snapmla_append_decode(c_kv_new, k_rope_new, n_new, q_nope, q_rope, kv_latent, kv_scale, k_rope, page_table,
                             seq_lens, B, q_len, H, max_pages, num_pages, page_size, softmax_scale, causal,
                             num_splits, kv_chunk_tokens, flags, ws, SNAPMLA_NOALLOC_SCRATCH_BYTES, out, out_dtype,
                             lse, stream);
  if (st != SNAPMLA_OK) return st;
  return snapmla_combine(ws, SNAPMLA_NOALLOC_SCRATCH_BYTES, seq_lens, B, q_len, H, num_splits, kv_chunk_tokens, out,
                         out_dtype, lse, stream);
}
