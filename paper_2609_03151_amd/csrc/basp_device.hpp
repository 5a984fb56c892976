// basp_device.hpp -- device-side helpers shared by the gfx950 kernels of
// libbasp: vector types, bf16 conversion, MFMA wrappers, lane exchange.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace basp {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two fp32 -> one dword holding {lo, hi} bf16 (lo in the low half), rounded
// to nearest even by the hardware packed conversion.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) {
  return __builtin_bit_cast(float, b << 16);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) {
  return __builtin_bit_cast(bf16x8, v);
}

// D = A * B + C on a 32x32 tile with a 16-deep bf16 contraction.
// Lane l supplies A[l%32][8*(l/32) .. +7] and B[8*(l/32) .. +7][l%32];
// the accumulator register r of lane l holds C[8*(r/4) + 4*(l/32) + r%4][l%32].
__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// 2^x on the hardware exp unit (no denormal fix-up needed for our ranges).
__device__ __forceinline__ float fast_exp2(float x) {
  return __builtin_amdgcn_exp2f(x);
}

__device__ __forceinline__ float fast_log2(float x) {
  return __builtin_amdgcn_logf(x);
}

// Value held by lane (l ^ 32).
__device__ __forceinline__ float swap_halves(float x) {
  return __shfl_xor(x, 32, kWave);
}

// Byte-select of two dwords: the low halves of a and b -> {a.lo, b.lo}.
__device__ __forceinline__ uint32_t lo_halves(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x05040100u);
}
// The high halves of a and b -> {a.hi, b.hi}.
__device__ __forceinline__ uint32_t hi_halves(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x07060302u);
}

// Position of key/row index j inside a 16-wide block when stored in the
// MFMA-operand order: swaps bits 2 and 3, so that lane half h reads the
// indices {4h..4h+3, 8+4h..8+4h+3} (what a 32x32 accumulator holds) as one
// contiguous 8-element run at [8h, 8h+8).
__device__ __forceinline__ int mfma_pos16(int j) {
  return (j & ~12) | ((j & 4) << 1) | ((j & 8) >> 1);
}

}  // namespace basp
