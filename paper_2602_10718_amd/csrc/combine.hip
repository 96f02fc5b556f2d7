// Split-KV log-sum-exp merge of the partial results of the decode kernel.
//
// Each KV piece p of a sequence delivered a normalized partial output o_p and its
// log-sum-exp LSE_p (Algorithm 1 returns both per query row).  Per row:
//   LSE = log sum_p exp(LSE_p),   o = sum_p exp(LSE_p - LSE) * o_p.
// One wave merges one row; lane l owns output dimensions 8l..8l+7.  The pieces'
// log-sum-exps are read lane-parallel and the partial rows four at a time.
// When the decode was given the output (ctrl[0] == 1) it has written the rows of
// every sequence that at most one piece covers; those are left as they are.

#include "piece_end.h"
#include "snapmla_device.h"
#include "snapmla_internal.h"

namespace snapmla {

__global__ __launch_bounds__(256) void combine_kernel(CombineArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t wv = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wv >= (int64_t)a.B * a.R) return;
  const int b = (int)(wv / a.R), r = (int)(wv % a.R);

  const int p0 = a.prefix[b], p1 = a.prefix[b + 1];
  const int nb = p1 - p0;
  const bool balanced = a.chunk_blocks == 0;
  const int64_t T = a.prefix[a.B];
  const int W = a.num_splits;
  // balanced plan: part w covers global blocks [w*T/W, (w+1)*T/W) and writes piece
  // id w + b for every sequence b it touches; fixed chunks: piece id b*W + chunk.
  // [first, last] is the candidate range; `exists` rejects empty parts.
  int first = 0, last = -1;
  if (nb > 0) {
    if (balanced) {
      first = (int)(((int64_t)(p0 + 1) * W - 1) / T);
      last = (int)(((int64_t)p1 * W - 1) / T);
    } else {
      first = 0;
      last = (nb + a.chunk_blocks - 1) / a.chunk_blocks - 1;
    }
  }
  // (a sequence with blocks meets only non-empty parts, so last - first + 1 is its
  // piece count)
  if (a.ctrl[0] == 1 && last <= first) return;
  auto exists = [&](int i) -> bool {
    if (!balanced) return true;
    return (int64_t)i * T / W < (int64_t)(i + 1) * T / W;
  };
  auto pid = [&](int i) -> int64_t { return balanced ? (int64_t)i + b : (int64_t)b * W + i; };

  // pass 1: lane i reads the log-sum-exp of candidate piece first + i (64 at a
  // time), the wave reduces the maximum and NaN flag
  float M = -INFINITY;
  bool anynan = false;
  for (int i0 = first; i0 <= last; i0 += 64) {
    const int i = i0 + lane;
    float x = -INFINITY;
    if (i <= last && exists(i)) x = a.part_lse[pid(i) * a.rows_pad + r];
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
        const float x = a.part_lse[pid(i) * a.rows_pad + r];
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

hipError_t launch_combine(const CombineArgs& a, hipStream_t stream) {
  const int64_t waves = (int64_t)a.B * a.R;
  if (waves <= 0) return hipSuccess;
  const int64_t blocks = (waves + 3) / 4;
  if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL(combine_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace snapmla
