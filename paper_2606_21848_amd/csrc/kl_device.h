// Device helpers shared by the keyless-attention kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kl {

typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// bf16 is carried as raw 16-bit words; two of them share a 32-bit register.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// c + a.lo * b.lo + a.hi * b.hi with bf16 inputs and an fp32 accumulator
// (one v_dot2c_f32_bf16).
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c, false);
}

// fp32 -> bf16, round to nearest even; NaN stays NaN.
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  return f32_to_bf16(lo) | (f32_to_bf16(hi) << 16);
}

// Lane permutation within rows of 16 lanes (DPP). CTRL: 0xB1 swaps neighbours,
// 0x4E swaps pairs, 0x141 mirrors each half row, 0x140 mirrors the row.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Sum over each aligned group of N consecutive lanes (N a power of two up to
// 32); every lane of the group receives the sum.
template <int N>
__device__ __forceinline__ float group_sum(float x) {
  if constexpr (N >= 2) x += dpp_f32<0xB1>(x);
  if constexpr (N >= 4) x += dpp_f32<0x4E>(x);
  if constexpr (N >= 8) x += dpp_f32<0x141>(x);
  if constexpr (N >= 16) x += dpp_f32<0x140>(x);
  if constexpr (N >= 32) x += __shfl_xor(x, 16);
  return x;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// One 16-byte-per-lane copy from global memory straight into LDS
// (global_load_lds_dwordx4): lane L's bytes land at lds + 16 L, where lds is a
// wave-uniform LDS byte address and gbase + voff the lane's source. Issued as
// inline assembly so the compiler does not serialise consecutive copies (it
// cannot tell they fill disjoint LDS rows). The copy counts against vmcnt:
// callers wait with s_waitcnt vmcnt and a barrier before the rows are read.
__device__ __forceinline__ void copy_to_lds(const void* gbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(gbase), "s"(lds)
               : "memory", "m0");
}

// The same copy with the non-temporal hint, for data streamed once.
__device__ __forceinline__ void copy_to_lds_nt(const void* gbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 nt"
               :
               : "v"(voff), "s"(gbase), "s"(lds)
               : "memory", "m0");
}

// s_waitcnt with only the vector-memory counter constrained (0..63).
#define KL_WAIT_VMCNT(n) \
  __builtin_amdgcn_s_waitcnt((((n) & 15) | (((n) >> 4) << 14)) | (0x7 << 4) | (0xF << 8))

// Merge two online-softmax states (m: running max in log2 units, l: sum of
// weights, a: weighted sum) into the first. An empty state has m = -inf, l = 0.
__device__ __forceinline__ void merge_scale(float m1, float m2, float& f1, float& f2, float& m) {
  m = fmaxf(m1, m2);
  const float ms = (m == -INFINITY) ? 0.f : m;
  f1 = fast_exp2(m1 - ms);
  f2 = fast_exp2(m2 - ms);
}

}  // namespace kl
