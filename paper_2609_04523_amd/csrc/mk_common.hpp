// mk_common.hpp -- device helpers shared by the gfx950 attention kernels.
//
// Register layouts of the CDNA4 matrix instructions used here (wave64):
//
//  v_mfma_f32_32x32x16_bf16  D[32x32] += A[32x16] * B[16x32]
//    A: lane l holds A[row = l%32][k-group l/32, 8 values]
//    B: lane l holds B[k-group l/32, 8 values][col = l%32]
//    D: lane l, register r holds D[row = 8*(r/4) + 4*(l/32) + r%4][col = l%32]
//
//  v_mfma_f32_16x16x32_bf16  D[16x16] += A[16x32] * B[32x16]
//    A: lane l holds A[row = l%16][k-group l/16, 8 values]
//    B: lane l holds B[k-group l/16, 8 values][col = l%16]
//    D: lane l, register r holds D[row = 4*(l/16) + r][col = l%16]
//
// A and B name their k-groups identically, so which 8 of the contraction
// indices a lane's k-group stands for is free, provided A and B agree.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mk {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.69314718055994531f;
constexpr float kNegInf = -__builtin_inff();

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// 2^x on the transcendental unit (v_exp_f32); 2^-inf = 0.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 u) { return __builtin_bit_cast(bf16x8, u); }
__device__ __forceinline__ u32x4 as_u32x4(bf16x8 b) { return __builtin_bit_cast(u32x4, b); }

// Eight fp32 -> eight bf16, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ bf16x8 to_bf16x8(float a0, float a1, float a2, float a3,
                                            float a4, float a5, float a6, float a7) {
  f32x8 f = {a0, a1, a2, a3, a4, a5, a6, a7};
  return __builtin_convertvector(f, bf16x8);
}

// fp32 -> bf16 bits, round to nearest even.
__device__ __forceinline__ uint16_t to_bf16_bits(float x) {
  __bf16 h = (__bf16)x;
  return __builtin_bit_cast(uint16_t, h);
}

// Value of lane (l ^ 32): the other half of the wave.
__device__ __forceinline__ float swap_halves(float x) {
  return __shfl_xor(x, 32, 64);
}

__device__ __forceinline__ int clamp_len(int len, int hi) {
  return len < 0 ? 0 : (len > hi ? hi : len);
}

}  // namespace mk
