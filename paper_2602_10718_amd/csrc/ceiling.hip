// Read-stream ceiling of the decode's page stream (a measurement kernel, not part
// of the attention path).  Every page of a list of 64-token blocks is moved into
// LDS by the same 16-byte direct-to-LDS loads the decode kernel uses, through a
// ring of the same depth (latent three blocks ahead in a 4-stage ring, RoPE and
// scales two ahead in a 3-stage ring), with no attention arithmetic.  Its time
// over the headline cache is the fastest any kernel of this copy structure can
// stream those pages, the "measured read-stream ceiling" the decode's bandwidth
// is reported against beside the 8 TB/s peak.
//
// So that the copies are observable, every thread XOR-folds one dword of each
// landed latent stage and one of each RoPE stage (dword tid: the first KiB of
// both), and each workgroup writes the XOR of its 256 threads: a checksum over
// the first KiB of latent and RoPE of every block of its range.

#include "snapmla_internal.h"
#include "snapmla_device.h"

namespace snapmla {

namespace {
constexpr int kCLat = 64 * 512;                 // latent bytes of a page
constexpr int kCRope = 64 * 64 * 2;             // RoPE bytes of a page
constexpr int kCSc = 64 * 4;                    // scale bytes of a page
constexpr int kCRs = kCRope + kCSc;             // RoPE + scales stage
constexpr int kCLatStages = 4, kCRsStages = 3;
constexpr int kCRsBase = kCLatStages * kCLat;
constexpr int kCIdBase = kCRsBase + kCRsStages * kCRs;
constexpr int kCSmem = kCIdBase + kCeilingMaxBlocks * 4;
static_assert(kCSmem <= 160 * 1024, "LDS budget of one workgroup");

// a wave-uniform pointer, kept in SGPRs for the scalar base operand of the copies
__device__ __forceinline__ const uint8_t* uniform_ptr(const uint8_t* p) {
  const uint64_t v = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<const uint8_t*>(((uint64_t)hi << 32) | lo);
}
}  // namespace

__global__ __launch_bounds__(256) void read_ceiling_kernel(CeilingArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t smem[kCSmem];
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int u = blockIdx.x;
  const int gs = (int)((int64_t)u * a.nblk / a.units), ge = (int)((int64_t)(u + 1) * a.nblk / a.units);
  const int n = ge - gs;                        // <= kCeilingMaxBlocks (checked by the host)
  int* ids = reinterpret_cast<int*>(smem + kCIdBase);
  // the range's page ids, by ordinary loads before any copy is in flight
  for (int i = tid; i < n; i += 256) {
    const int p = a.pages[gs + i];
    ids[i] = (p >= 0 && p < a.num_pages) ? p : 0;
  }
  __syncthreads();
  if (n <= 0) {
    if (tid == 0) a.out[u] = 0u;
    return;
  }
  const uint32_t base = lds_offset(smem);
  // blocks past the range repeat the last page into the stage they would take,
  // which nothing reads; so every period issues the same copies and the waits
  // below are exact
  auto page_of = [&](int j) { return __builtin_amdgcn_readfirstlane(ids[j < n ? j : n - 1]); };
  // wave w copies latent rows 16w..16w+15 (8 KiB, eight 1 KiB loads), RoPE rows
  // 16w..16w+15 (2 KiB, two loads) and scales 16w..16w+15 (lanes 0-15, 4 bytes each)
  auto copy_lat = [&](int j) {
    const uint8_t* src = a.kv_latent + (int64_t)page_of(j) * kCLat + 8192 * w;
    const uint32_t dst = base + (j % kCLatStages) * kCLat + 8192 * w;
#pragma unroll
    for (int i = 0; i < 8; ++i) g2lds16_so(src + 1024 * i, (uint32_t)(16 * lane), dst + 1024 * i);
  };
  auto copy_rs = [&](int j) {
    const int p = page_of(j);
    const uint8_t* rp = reinterpret_cast<const uint8_t*>(a.k_rope) + (int64_t)p * kCRope + 2048 * w;
    const uint8_t* sp = uniform_ptr(reinterpret_cast<const uint8_t*>(a.kv_scale) + (int64_t)p * kCSc + 64 * w);
    const uint32_t dst = base + kCRsBase + (j % kCRsStages) * kCRs;
#pragma unroll
    for (int i = 0; i < 2; ++i) g2lds16_so(rp + 1024 * i, (uint32_t)(16 * lane), dst + 2048 * w + 1024 * i);
    if (lane < 16) g2lds4_so(sp, (uint32_t)(4 * lane), dst + kCRope + 64 * w);
  };
  // prologue, in issue order: latent 0, RoPE 0, latent 1, RoPE 1, latent 2
  copy_lat(0);
  copy_rs(0);
  copy_lat(1);
  copy_rs(1);
  copy_lat(2);
  uint32_t acc = 0u;
  for (int k = 0; k < n; ++k) {
    // block k landed: in issue order its RoPE copy is followed by the latent copy
    // of block k+1 (8) and the 11 copies of the previous period (in period 0 by
    // RoPE 1 and latent 2 of the prologue): at most 19 outstanding
    barrier_vm_lgkm0<19>();
    acc ^= *reinterpret_cast<const uint32_t*>(smem + (k % kCLatStages) * kCLat + 4 * tid);
    acc ^= *reinterpret_cast<const uint32_t*>(smem + kCRsBase + (k % kCRsStages) * kCRs + 4 * tid);
    // the stages of block k-1, read in the previous period, take blocks k+2 / k+3
    copy_rs(k + 2);
    copy_lat(k + 3);
  }
  barrier_vm_lgkm0<0>();                        // no copy may land after the workgroup ends
  acc ^= __shfl_xor(acc, 32);
  acc ^= __shfl_xor(acc, 16);
  acc ^= __shfl_xor(acc, 8);
  acc ^= __shfl_xor(acc, 4);
  acc ^= __shfl_xor(acc, 2);
  acc ^= __shfl_xor(acc, 1);
  uint32_t* red = reinterpret_cast<uint32_t*>(smem + kCIdBase);
  if (lane == 0) red[w] = acc;
  __syncthreads();
  if (tid == 0) a.out[u] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

hipError_t launch_read_ceiling(const CeilingArgs& a, hipStream_t stream) {
  if (a.units <= 0) return hipSuccess;
  hipLaunchKernelGGL(read_ceiling_kernel, dim3((unsigned)a.units), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace snapmla

namespace snapmla {

// Plain read stream (a measurement kernel): the buffer read once with 16-byte
// vector loads, a grid-stride loop over 16-byte words with consecutive lanes on
// consecutive words, each thread XOR-folding what it read; each workgroup
// writes the XOR of its 256 threads.  No LDS, no copies: the rate the memory
// system gives a simple streaming kernel, the second reference figure beside
// the 8 TB/s peak.
__global__ __launch_bounds__(256) void read_stream_kernel(const v4i* __restrict__ p, int64_t n16, uint32_t* out) {
  __shared__ uint32_t red[4];
  v4i acc = {0, 0, 0, 0};
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += stride) acc ^= p[i];
  uint32_t x = (uint32_t)(acc[0] ^ acc[1] ^ acc[2] ^ acc[3]);
  x ^= __shfl_xor(x, 32);
  x ^= __shfl_xor(x, 16);
  x ^= __shfl_xor(x, 8);
  x ^= __shfl_xor(x, 4);
  x ^= __shfl_xor(x, 2);
  x ^= __shfl_xor(x, 1);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) out[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

hipError_t launch_read_stream(const void* buf, int64_t n16, int grid, uint32_t* out, hipStream_t stream) {
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL(read_stream_kernel, dim3((unsigned)grid), dim3(256), 0, stream,
                     static_cast<const v4i*>(buf), n16, out);
  return hipGetLastError();
}

}  // namespace snapmla
