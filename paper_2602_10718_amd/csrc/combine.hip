// Split-KV log-sum-exp merge of the partial results of the decode kernel.
//
// Each KV piece p of a sequence delivered a normalized partial output o_p and its
// log-sum-exp LSE_p (Algorithm 1 returns both per query row).  Per row:
//   LSE = log sum_p exp(LSE_p),   o = sum_p exp(LSE_p - LSE) * o_p.
// When the decode was given the output (ctrl[0] == 1) it has written the rows of
// every sequence that at most one piece covers; those are left as they are.
//
// Two kernels, one per slot layout (part_tile_offset):
// - one row group (plain rows): one wave per row; lane l owns output dimensions
//   8l..8l+7.  The pieces' log-sum-exps are read lane-parallel, and a piece whose
//   weight underflows to zero is not read at all (the row's partial sits in its own
//   cache lines).
// - several row groups (tile order): one wave per 32-row x 32-dimension tile, lane
//   n + 32h on row n of the tile, dimensions 8q + 4h .. +3; every partial load of a
//   wave reads 1 KiB of consecutive bytes.  Each lane merges its row with a running
//   maximum, four pieces per round so that their loads overlap.

#include "piece_end.h"
#include "snapmla_device.h"
#include "snapmla_internal.h"

namespace snapmla {

// The pieces of sequence b: candidates first..last; exists(i) rejects an empty part
// (only possible with fewer virtual positions than parts), pid(i) is the piece's slot.
// Balanced plan: part w covers the real blocks of virtual positions [w*TV/W,
// (w+1)*TV/W) (kPlanPad) and writes piece id w + b for every sequence b it touches;
// fixed chunks: piece id b*W + chunk.  (The parts that meet sequence b's real blocks
// are exactly those whose virtual range meets [prefix[b] + pad*(b+1), prefix[b+1] +
// pad*(b+1)); each of them has a non-empty range, so last - first + 1 counts its pieces.)
struct Pieces {
  int first = 0, last = -1, b = 0, W = 1;
  bool balanced = true;
  int64_t TV = 0;
  __device__ bool exists(int i) const {
    return !balanced || TV >= W || (int64_t)i * TV / W < (int64_t)(i + 1) * TV / W;
  }
  __device__ int64_t pid(int i) const { return balanced ? (int64_t)i + b : (int64_t)b * W + i; }
};

__device__ Pieces pieces_of(const CombineArgs& a, int b) {
  Pieces P;
  P.b = b;
  P.W = a.num_splits;
  P.balanced = a.chunk_blocks == 0;
  P.TV = a.prefix[a.B] + (int64_t)a.pad * a.B;
  const int p0 = a.prefix[b], p1 = a.prefix[b + 1];
  const int nb = p1 - p0;
  if (nb > 0) {
    if (P.balanced) {
      const int64_t v0 = p0 + (int64_t)a.pad * (b + 1);    // virtual position of the first block
      P.first = (int)(((v0 + 1) * P.W - 1) / P.TV);
      P.last = (int)(((v0 + nb) * P.W - 1) / P.TV);
    } else {
      P.first = 0;
      P.last = (nb + a.chunk_blocks - 1) / a.chunk_blocks - 1;
    }
  }
  return P;
}

__global__ __launch_bounds__(256) void combine_rows_kernel(CombineArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t wv = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wv >= (int64_t)a.B * a.R) return;
  const int b = (int)(wv / a.R), r = (int)(wv % a.R);

  const Pieces P = pieces_of(a, b);
  const int first = P.first, last = P.last;
  if (a.ctrl[0] == 1 && last <= first) return;
  auto exists = [&](int i) { return P.exists(i); };
  auto pid = [&](int i) { return P.pid(i); };

  // pass 1: lane i reads the log-sum-exp of candidate piece first + i (64 at a
  // time), the wave reduces the maximum and NaN flag; the first 64 stay in x0 for
  // pass 2
  float M = -INFINITY;
  bool anynan = false;
  float x0 = -INFINITY;
  for (int i0 = first; i0 <= last; i0 += 64) {
    const int i = i0 + lane;
    float x = -INFINITY;
    if (i <= last && exists(i)) x = a.part_lse[pid(i) * a.rows_pad + r];
    if (i0 == first) x0 = x;
    anynan |= x != x;
    M = fmaxf(M, x);
  }
  M = wave_max(M);
  anynan = __builtin_amdgcn_ballot_w64(anynan) != 0;
  // pass 2: weights exp(LSE_i - M) (lane-parallel), then the weighted rows, four
  // pieces per round so that their loads overlap
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  float S = 0.0f;
  if (M > -INFINITY && !anynan) {
    for (int i0 = first; i0 <= last; i0 += 64) {
      const int i = i0 + lane;
      float wi = 0.0f;
      if (i <= last && exists(i)) {
        const float x = i0 == first ? x0 : a.part_lse[pid(i) * a.rows_pad + r];
        wi = x > -INFINITY ? expf(x - M) : 0.0f;
      }
      S += wi;
      const int cnt = min(64, last - i0 + 1);
      for (int j = 0; j < cnt; j += 4) {
        v4f u[4][2];
        float wj[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          wj[t] = __shfl(wi, j + t, 64);              // zero for missing / empty pieces
          const bool use = j + t < cnt && wj[t] != 0.0f;
          const int ij = min(i0 + j + t, last);      // in range even when unused
          const v4f* src = reinterpret_cast<const v4f*>(a.part_o + (pid(ij) * a.rows_pad + r) * kDc + 8 * lane);
          u[t][0] = use ? src[0] : v4f{0.f, 0.f, 0.f, 0.f};
          u[t][1] = use ? src[1] : v4f{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          acc[0] += wj[t] * u[t][0][0]; acc[1] += wj[t] * u[t][0][1];
          acc[2] += wj[t] * u[t][0][2]; acc[3] += wj[t] * u[t][0][3];
          acc[4] += wj[t] * u[t][1][0]; acc[5] += wj[t] * u[t][1][1];
          acc[6] += wj[t] * u[t][1][2]; acc[7] += wj[t] * u[t][1][3];
        }
      }
    }
    // wave sum of the weights
    for (int o = 32; o > 0; o >>= 1) S += __shfl_xor(S, o, 64);
  }
  const bool bad = a.flags[b] != 0 || anynan;
  float o[8];
  float lse;
  if (bad) {
    const float nanv = __builtin_nanf("");
    for (int j = 0; j < 8; ++j) o[j] = nanv;
    lse = nanv;
  } else if (!(M > -INFINITY)) {
    for (int j = 0; j < 8; ++j) o[j] = 0.0f;
    lse = -INFINITY;
  } else {
    const float inv = 1.0f / S;
    for (int j = 0; j < 8; ++j) o[j] = acc[j] * inv;
    lse = M + logf(S);
  }
  const int64_t orow = (int64_t)b * a.R + r;
  if (a.out_dtype == 1) {
    v4f* dst = reinterpret_cast<v4f*>(reinterpret_cast<float*>(a.out) + orow * kDc + 8 * lane);
    dst[0] = v4f{o[0], o[1], o[2], o[3]};
    dst[1] = v4f{o[4], o[5], o[6], o[7]};
  } else {
    uint4 pk;
    pk.x = f32_to_bf16_bits(o[0]) | (f32_to_bf16_bits(o[1]) << 16);
    pk.y = f32_to_bf16_bits(o[2]) | (f32_to_bf16_bits(o[3]) << 16);
    pk.z = f32_to_bf16_bits(o[4]) | (f32_to_bf16_bits(o[5]) << 16);
    pk.w = f32_to_bf16_bits(o[6]) | (f32_to_bf16_bits(o[7]) << 16);
    reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(a.out) + orow * kDc)[lane] = pk;
  }
  if (a.lse != nullptr && lane == 0) a.lse[orow] = lse;
}

__global__ __launch_bounds__(256) void combine_tiles_kernel(CombineArgs a) {
  const int lane = threadIdx.x & 63;
  const int n = lane & 31, h = lane >> 5;
  const int T = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tiles = (a.R + 31) / 32;                 // 32-row tiles per sequence
  const int dq = (int)(blockIdx.x & 3);
  const int64_t bt = blockIdx.x >> 2;
  const int b = (int)(bt / tiles), t = (int)(bt % tiles);
  const int row = 32 * t + n;                        // query row of this lane (< rows_pad)

  const Pieces P = pieces_of(a, b);
  const int first = P.first, last = P.last;
  if (a.ctrl[0] == 1 && last <= first) return;
  auto exists = [&](int i) { return P.exists(i); };
  auto pid = [&](int i) { return P.pid(i); };
  const int64_t tile = part_tile_offset(t >> 1, dq, t & 1, T, 0, lane);

  // this wave's pieces, merged with a running maximum M: S = sum exp(LSE_i - M),
  // acc = sum exp(LSE_i - M) o_i.  Every row of an existing piece's slot was written
  // (0 for a row without tokens, NaN for a rejected piece).
  float M = -INFINITY, S = 0.0f;
  bool anynan = false;
  v4f acc[4] = {v4f{0.f, 0.f, 0.f, 0.f}, v4f{0.f, 0.f, 0.f, 0.f}, v4f{0.f, 0.f, 0.f, 0.f}, v4f{0.f, 0.f, 0.f, 0.f}};
  for (int i0 = first; i0 <= last; i0 += 4) {
    float x[4];
    v4f u[4][4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = i0 + j;
      const bool live = i <= last && exists(i);
      const int64_t p = pid(live ? i : first);       // in range even when unused
      x[j] = live ? a.part_lse[p * a.rows_pad + row] : -INFINITY;
      const v4f* src = reinterpret_cast<const v4f*>(a.part_o + p * a.rows_pad * kDc + tile);
#pragma unroll
      for (int q = 0; q < 4; ++q) u[j][q] = live ? src[64 * q] : v4f{0.f, 0.f, 0.f, 0.f};
    }
    float mr = M;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      anynan |= x[j] != x[j];
      mr = fmaxf(mr, x[j]);
    }
    if (mr > -INFINITY) {
      const float sc = expf(M - mr);                 // 0 while M is -inf
      S *= sc;
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[q] *= sc;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float wj = x[j] > -INFINITY ? expf(x[j] - mr) : 0.0f;
        S += wj;
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[q] += wj * u[j][q];
      }
      M = mr;
    }
  }
  if (row >= a.R) return;
  const bool bad = a.flags[b] != 0 || anynan;
  v4f o[4];
  float lse;
  if (bad) {
    const float nanv = __builtin_nanf("");
    for (int q = 0; q < 4; ++q) o[q] = v4f{nanv, nanv, nanv, nanv};
    lse = nanv;
  } else if (!(M > -INFINITY)) {
    for (int q = 0; q < 4; ++q) o[q] = v4f{0.f, 0.f, 0.f, 0.f};
    lse = -INFINITY;
  } else {
    const float inv = 1.0f / S;
    for (int q = 0; q < 4; ++q) o[q] = acc[q] * inv;
    lse = M + logf(S);
  }
  const int64_t orow = (int64_t)b * a.R + row;
  const int64_t col = 128 * dq + 32 * T + 4 * h;
  for (int q = 0; q < 4; ++q) {
  if (a.out_dtype == 1) {
    *reinterpret_cast<v4f*>(reinterpret_cast<float*>(a.out) + orow * kDc + col + 8 * q) = o[q];
  } else {
    const uint32_t lo = f32_to_bf16_bits(o[q][0]) | (f32_to_bf16_bits(o[q][1]) << 16);
    const uint32_t hi = f32_to_bf16_bits(o[q][2]) | (f32_to_bf16_bits(o[q][3]) << 16);
    *reinterpret_cast<v2i*>(reinterpret_cast<uint16_t*>(a.out) + orow * kDc + col + 8 * q) = v2i{(int)lo, (int)hi};
  }
  }
  if (a.lse != nullptr && dq == 0 && T == 0 && h == 0) a.lse[orow] = lse;
}

hipError_t launch_combine(const CombineArgs& a, hipStream_t stream) {
  if ((int64_t)a.B * a.R <= 0) return hipSuccess;
  if (a.rows_pad > 64) {
    // one workgroup per sequence, 32-row tile and 128-dimension quarter
    const int64_t blocks = (int64_t)a.B * ((a.R + 31) / 32) * 4;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL(combine_tiles_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a);
  } else {
    const int64_t blocks = ((int64_t)a.B * a.R + 3) / 4;   // one wave per row
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL(combine_rows_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace snapmla
