// Device helpers shared by the masked-MoE kernels (gfx950 / CDNA4, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace maskmoe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));  // one 16-byte load / LDS access

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// float -> bf16 bits, round to nearest even; a NaN keeps its sign and upper payload bits and
// becomes quiet. gfx950 converts in one instruction (v_cvt_pk_bf16_f32, two values at a
// time); it matches the bit-level rounding (add 0x7fff plus the kept lsb, NaN -> bits | 0x40)
// on all 2^32 inputs, and takes no branch for the NaN case.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t f32x2_to_bf16x2(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

// D = A(16x32) * B(32x16) + C on bf16 operands, fp32 accumulate.
// Operand layout per lane l: A row (l & 15), B column (l & 15), eight consecutive k values
// at k-group (l >> 4); the same k-group assignment is used for A and B.
// Result layout: lane l holds column (l & 15), rows 4 * (l >> 4) + i, i = 0..3.
__device__ __forceinline__ f32x4 mfma_16x16x32(const u32x4& a, const u32x4& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                  __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// D = A(32x16) * B(16x32) + C on bf16 operands, fp32 accumulate.
// Operand layout per lane l: A row (l & 31), B column (l & 31), eight consecutive k values
// at k-group (l >> 5). Result layout: lane l holds column (l & 31) and, for acc index
// r = 4 * j + i, row 8 * j + 4 * (l >> 5) + i.
__device__ __forceinline__ f32x16 mfma_32x32x16(const u32x4& a, const u32x4& b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                  __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// silu(u) = u sigmoid(u); the hardware reciprocal (1 ulp) instead of an IEEE division: the
// result is rounded to bf16 next, and the division's scale-and-fix-up sequence was most of
// the gate/up epilogue's arithmetic.
__device__ __forceinline__ float sigmoid(float u) { return __builtin_amdgcn_rcpf(1.0f + __expf(-u)); }
__device__ __forceinline__ float silu(float u) { return u * sigmoid(u); }

__device__ __forceinline__ int wave_min_int(int v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = min(v, __shfl_xor(v, m, kWave));
  return v;
}

__device__ __forceinline__ int wave_sum_int(int v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}

__device__ __forceinline__ uint64_t lanemask_lt(int lane) {
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Workgroup barrier ordering LDS accesses only. __syncthreads() also waits until every global
// store the thread has issued is acknowledged, which costs a memory round trip after a kernel
// writes outputs; where threads exchange data through LDS alone, this one waits for LDS only.
__device__ __forceinline__ void lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// XOR swizzle of the eight 16-byte chunks of a 128-byte LDS operand row: row bits 0..2, with
// row bit 3 flipping chunk bit 0. A 16-byte operand read whose lanes walk 16 consecutive rows
// at one logical chunk then touches 16 distinct bank groups, for 32 or 64 four-byte banks; rows
// 64 apart share the swizzle term.
__device__ __forceinline__ int lds_swizzle(int row) { return (row & 7) ^ ((row >> 3) & 1); }

}  // namespace maskmoe
