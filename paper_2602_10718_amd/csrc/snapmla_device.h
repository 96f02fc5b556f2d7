// Device-side building blocks shared by the SnapMLA kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace snapmla {

// Shapes fixed by the method: 512-d content latent, 64-d RoPE part (Section 3.1:
// eight content groups of 64 plus one RoPE group), 64-token pages that are also the
// probability-quantization blocks (Section 3.2 (ii), BlockN = 64).
constexpr int kDc = 512;
constexpr int kDr = 64;
constexpr int kPage = 64;
constexpr float kFp8Max = 448.0f;
// floor of every dynamic scale (Appendix D lower-bounds scales by a small epsilon)
constexpr float kEps = 9.094947017729282e-13f;  // 2^-40

typedef int v2i __attribute__((ext_vector_type(2)));
typedef float v2f __attribute__((ext_vector_type(2)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef short v8s __attribute__((ext_vector_type(8)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v2i lds_v2i;

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// OCP E4M3 encode of two floats into bytes 0/1 (hi=false) or 2/3 (hi=true) of `old`.
// The hardware conversion rounds to nearest even; inputs must stay below 464 in
// magnitude (callers clamp where that is not guaranteed by construction).
__device__ __forceinline__ int cvt_pk_e4m3(float a, float b, int old, bool hi) {
  return hi ? __builtin_amdgcn_cvt_pk_fp8_f32(a, b, old, true)
            : __builtin_amdgcn_cvt_pk_fp8_f32(a, b, old, false);
}

__device__ __forceinline__ float clamp448(float x) { return fminf(fmaxf(x, -kFp8Max), kFp8Max); }

// 16x16x128 FP8 MFMA: lane (i%16, i/16) holds A[i%16][32*(i/16) + 0..31] and
// B[32*(i/16) + 0..31][i%16]; C lane i register v is C[4*(i/16) + v][i%16].
__device__ __forceinline__ v4f mfma_f8_16x16x128(v8i a, v8i b, v4f c) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// 16x16x32 F16 MFMA: lane (i%16, i/16) holds K = 8*(i/16) + 0..7; same C layout.
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
__device__ __forceinline__ v4f mfma_f16_16x16x32(v4i a, v4i b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(v8h, a), __builtin_bit_cast(v8h, b), c, 0, 0, 0);
}

// Four E4M3 codes (bytes of one dword) -> four halfs in two dwords.  The conversion
// is exact: every E4M3 value, subnormals included, is a normal f16 value.
__device__ __forceinline__ v2i e4m3x4_to_f16(int x) {
  const auto lo = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8((unsigned)x, 1.0f, false);
  const auto hi = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8((unsigned)x, 1.0f, true);
  return v2i{__builtin_bit_cast(int, lo), __builtin_bit_cast(int, hi)};
}
// Eight codes (two dwords) -> the eight-half operand of one 16x16x32 F16 MFMA.
__device__ __forceinline__ v4i e4m3x8_to_f16(int x0, int x1) {
  const v2i a = e4m3x4_to_f16(x0), b = e4m3x4_to_f16(x1);
  return v4i{a[0], a[1], b[0], b[1]};
}

// 16x16x32 BF16 MFMA: lane (i%16, i/16) holds K = 8*(i/16) + 0..7; same C layout.
__device__ __forceinline__ v4f mfma_bf16_16x16x32(v4i a, v4i b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a), __builtin_bit_cast(v8bf, b), c, 0, 0, 0);
}

// 32x32x64 FP8 (E4M3 x E4M3) MFMA, float32 accumulate.  Lane (i%32, i/32) holds
// A[i%32][32*(i/32) + 0..31] and B[32*(i/32) + 0..31][i%32]; C lane i register v is
// C[8*(v/4) + 4*(i/32) + v%4][i%32].
__device__ __forceinline__ v16f mfma_f8_32x32x64(v8i a, v8i b, v16f c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// 32x32x16 BF16 MFMA: lane (i%32, i/32) holds K = 8*(i/32) + 0..7; same C layout.
__device__ __forceinline__ v16f mfma_bf16_32x32x16(v4i a, v4i b, v16f c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, a),
                                                 __builtin_bit_cast(v8bf, b), c, 0, 0, 0);
}

// Maximum / sum across the two 32-lane halves (lane i and lane i^32).
__device__ __forceinline__ float xhalf_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xhalf_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Maximum / sum over the four lanes i, i^16, i^32, i^48 (one row of a 16x16 tile).
__device__ __forceinline__ float quad_max(float x) {
  x = xhalf_max(x);
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float quad_sum(float x) {
  x = xhalf_sum(x);
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// The same maximum with NaN-propagating semantics (v_maximum3_f32 on gfx950): no
// quieting of signalling NaNs is needed first, so reductions over values the compiler
// cannot prove canonical (lane swaps, merged branches) take one instruction per pair
// or triple.  For callers whose inputs hold no NaN (masked slots are -inf), the result
// equals fmaxf's.
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }
__device__ __forceinline__ float vmax3(float a, float b, float c) { return vmax(vmax(a, b), c); }
__device__ __forceinline__ float quad_vmax(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = vmax(__uint_as_float(r[0]), __uint_as_float(r[1]));
  r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return vmax(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
// max over 16 values as five three-input maxima
__device__ __forceinline__ float vmax16(const float (&v)[16]) {
  const float a = vmax3(v[0], v[1], v[2]), b = vmax3(v[3], v[4], v[5]), c = vmax3(v[6], v[7], v[8]);
  const float d = vmax3(v[9], v[10], v[11]), e = vmax3(v[12], v[13], v[14]);
  return vmax(vmax3(a, b, c), vmax3(d, e, v[15]));
}

__device__ __forceinline__ float wave_max(float x) {
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] at [15:14]).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Workgroup barrier that waits only for what the caller names: the vector-memory
// counter down to VM (direct-to-LDS copies still in flight may stay in flight)
// and all LDS operations of this wave.  The empty asm statements keep the
// compiler from moving memory accesses across the barrier.  (__syncthreads()
// would also drain every outstanding direct-to-LDS copy.)
template <int VM>
__device__ __forceinline__ void barrier_vm_lgkm0() {
  static_assert(VM >= 0 && VM < 64, "vmcnt range");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((VM & 0xF) | ((VM >> 4) << 14) | (0x7 << 4));   // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// 16-byte (or 4-byte) global -> LDS copy: lane i writes its bytes at lds_base + i*size
// (lds_base must be wave-uniform).  Written as inline assembly on purpose: the
// compiler's own form of this instruction makes it drain every outstanding copy
// before each later LDS transpose read (it cannot tell which LDS bytes a copy
// writes).  The kernels wait for these copies explicitly with s_waitcnt vmcnt.
__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return (uint32_t)(uintptr_t)((__attribute__((address_space(3))) const uint8_t*)p);
}
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void g2lds16(const void* gptr, void* lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
               :: "s"(__builtin_amdgcn_readfirstlane(lds_offset(lds_base))), "v"(gptr) : "memory", "m0");
}
__device__ __forceinline__ void g2lds4(const void* gptr, void* lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, off"
               :: "s"(__builtin_amdgcn_readfirstlane(lds_offset(lds_base))), "v"(gptr) : "memory", "m0");
}
// Same copies addressed as a wave-uniform 64-bit base (SGPRs) plus a per-lane
// 32-bit byte offset, so the address costs no vector instructions.
__device__ __forceinline__ void g2lds16_so(const void* sbase, uint32_t voff, uint32_t lds_off) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
               :: "s"(__builtin_amdgcn_readfirstlane(lds_off)), "v"(voff), "s"(sbase) : "memory", "m0");
}
__device__ __forceinline__ void g2lds4_so(const void* sbase, uint32_t voff, uint32_t lds_off) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, %2"
               :: "s"(__builtin_amdgcn_readfirstlane(lds_off)), "v"(voff), "s"(sbase) : "memory", "m0");
}
#pragma clang diagnostic pop

// Returns x unchanged but opaque to the optimiser, so that per-iteration address
// arithmetic is not hoisted out of a software-pipelined loop (where the hoisted
// values would only be spilled).
__device__ __forceinline__ uint32_t opaque_u32(uint32_t x) {
  asm volatile("" : "+v"(x));
  return x;
}
// The same for a wave-uniform value, kept in a scalar register.
__device__ __forceinline__ uint32_t opaque_s32(uint32_t x) {
  x = __builtin_amdgcn_readfirstlane(x);
  asm volatile("" : "+s"(x));
  return x;
}

__device__ __forceinline__ v2i lds_read_tr8(const uint8_t* p) {
  return __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_v2i*)(p));
}
// Same read addressed by a 32-bit LDS byte address.
__device__ __forceinline__ v2i lds_read_tr8_at(uint32_t lds_addr) {
  return __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_v2i*)(uintptr_t)lds_addr);
}

}  // namespace snapmla
