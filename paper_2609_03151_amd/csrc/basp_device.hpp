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

typedef short i16x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- buffers
// Raw buffer resource over [base, base + num_bytes): loads whose offset falls
// outside return zeros without touching memory, which handles ragged tails
// without branches.  Offsets are 32-bit (num_bytes < 2^31, checked on the
// host).  Word 3 selects the 32-bit data format expected by raw loads.
typedef __amdgpu_buffer_rsrc_t rsrc_t;

__device__ __forceinline__ rsrc_t make_rsrc(const void *base, uint32_t num_bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)num_bytes,
                                           0x00020000);
}
__device__ __forceinline__ u32x4 buf_load16(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

// 16 bytes per lane from buffer offset `off` straight into LDS, bypassing
// registers: lane l's bytes land at lds_addr + 16*l.  Out-of-range offsets
// write zeros.  Completion is counted by vmcnt like any buffer load.
// Issued through inline asm: the compiler then does not know the
// instruction writes LDS, so it neither holds later LDS reads back until
// every copy in flight has landed (which would drain a prefetch ring) nor
// orders anything against it.  The caller waits (vmcnt) for its own copies
// and passes a barrier before any wave reads the data.  `rsrc` and
// `lds_addr` (an LDS byte address, passed in M0) must be wave-uniform.  One
// wait state separates the compiler's M0 write from the load.
__device__ __forceinline__ void buf_load16_lds_async(u32x4 rsrc, uint32_t off, uint32_t lds_addr) {
  asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
               :
               : "v"(off), "s"(rsrc), "{m0}"(lds_addr)
               : "memory");
}

// Raw buffer descriptor as four dwords (same fields make_rsrc sets): base
// address, stride 0, size in bytes, 32-bit data format.
__device__ __forceinline__ u32x4 make_rsrc_words(const void *base, uint32_t num_bytes) {
  const uint64_t a = (uint64_t)(uintptr_t)base;
  return u32x4{(uint32_t)a, (uint32_t)(a >> 32) & 0xFFFFu, num_bytes, 0x00020000u};
}

// LDS byte address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_addr_of(const void *p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)p;
}

// Workgroup barrier without the memory fence __syncthreads() adds (that
// fence waits for every outstanding global load, including prefetches).
// The empty asm statements keep the compiler from moving memory accesses
// across it; visibility of LDS copies is the caller's explicit vmcnt wait.
__device__ __forceinline__ void barrier_no_fence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// max and sum of the values held by lanes l and l^32, in both lanes.
// v_permlane32_swap exchanges lanes 32-63 of its first register with lanes
// 0-31 of its second; with both holding x, the first ends up holding the
// lower half of x in both halves and the second the upper half.  (Issued as
// inline asm: the compiler builtin loses its second result.)  The nops
// cover the VALU-write -> permlane-read hazard and the one after it.
__device__ __forceinline__ void lane_halves(float x, float &lo, float &hi) {
  lo = x;
  hi = x;
  asm("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(lo), "+v"(hi));
}
__device__ __forceinline__ float pair_max(float x) {
  float lo, hi;
  lane_halves(x, lo, hi);
  return fmaxf(lo, hi);
}
__device__ __forceinline__ float pair_sum(float x) {
  float lo, hi;
  lane_halves(x, lo, hi);
  return lo + hi;
}

// Issue priority of this wave on its SIMD (s_setprio, 0 = default).  The
// two waves that share a SIMD run the same tile loop side by side; raising
// the priority over one block of MFMAs lets whichever wave gets there first
// keep the matrix unit while the other does its VALU work, instead of both
// alternating through both phases.  Scheduling barriers keep the compiler
// from moving instructions across the switch.
template <int P>
__device__ __forceinline__ void wave_priority() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_setprio(P);
  __builtin_amdgcn_sched_barrier(0);
}

// s_waitcnt vmcnt(n) with the other counters left alone (n < 64).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}

// ------------------------------------------------------------- LDS tiles
// A [rows][D] bf16 tile stored row-major without padding, its 16-byte chunks
// permuted by an XOR of the row (a key that depends on the row modulo 16).
// With LDS serving 256 bytes per cycle, the permutation makes both access
// patterns of the attention kernels free of bank conflicts:
//   * 16 lanes reading one chunk of 16 consecutive rows (MFMA operand rows):
//     the key is a bijection on the 16 rows;
//   * 32 lanes of ds_read_b64_tr_b16 reading 4 consecutive rows, starting at
//     a multiple of 4, at 4 consecutive chunks starting at a multiple of 4:
//     the keys of those rows differ in their upper bits, so the 16 chunk
//     slots they touch are distinct.
template <int D>
struct LdsTile;

template <>
struct LdsTile<128> {
  static constexpr int ROW_BYTES = 256;
  __device__ static __forceinline__ int swz(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }
  __device__ static __forceinline__ int off(int r, int chunk) {
    return r * ROW_BYTES + ((chunk ^ swz(r)) << 4);
  }
};

template <>
struct LdsTile<64> {
  static constexpr int ROW_BYTES = 128;
  __device__ static __forceinline__ int swz(int r) {
    return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
  }
  __device__ static __forceinline__ int off(int r, int chunk) {
    return r * ROW_BYTES + ((chunk ^ swz(r)) << 4);
  }
};

// Head dims the attention kernels take, with the width their MFMA tiles
// compute at (DC, a multiple of 32) and the LDS row layout they use (LW):
// 80 and 96 compute at 96, kept in the 128-wide layout; the columns past D
// are zeros everywhere they enter a product.
template <int D>
struct HeadDim;
template <>
struct HeadDim<64> {
  static constexpr int DC = 64, LW = 64;
};
template <>
struct HeadDim<80> {
  static constexpr int DC = 96, LW = 128;
};
template <>
struct HeadDim<96> {
  static constexpr int DC = 96, LW = 128;
};
template <>
struct HeadDim<128> {
  static constexpr int DC = 128, LW = 128;
};

// A buffer offset no resource of the library reaches (ranges stay below
// 2^31): loads from it return zeros.
constexpr uint32_t kZeroOffset = 0x80000000u;

// Source offset, within a tile of rows `row_bytes` apart in memory, of the
// 16-byte chunk that a linear LDS copy places at chunk slot `pos` of an
// LdsTile<LW>: slot pos holds row pos / (LW/8), stored chunk pos % (LW/8),
// i.e. logical chunk (stored chunk) ^ swz(row).  Copying chunk slots in order
// with buf_load16_lds_async therefore leaves the tile in its swizzled layout.
// Logical chunks past the row's D elements read from kZeroOffset, so the
// padding columns of the tile are zeros.
template <int LW, int D = LW>
__device__ __forceinline__ uint32_t dma_src_off(int pos, uint32_t row_bytes) {
  constexpr int CPR = LW / 8;
  const int r = pos / CPR, pc = pos % CPR;
  const int lc = pc ^ LdsTile<LW>::swz(r);
  if (D < LW && lc >= D / 8) return kZeroOffset;
  return (uint32_t)r * row_bytes + (lc << 4);
}

typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// ds_read_b64_tr_b16: each lane passes the address of 4 consecutive bf16; in
// every group of 16 lanes, lane i receives element i%4 of the 8-byte pieces
// addressed by lanes i/4, i/4+4, i/4+8, i/4+12.  With lane c of the group
// addressing row r0 + c/4, columns e0 + 4(c%4) .. +3, lane i therefore gets
// the column e0 + i over rows r0 .. r0+3: a transposed read.  Two such reads
// give one MFMA operand (slots 0-3 and 4-7).
__device__ __forceinline__ bf16x8 tr_operand(const unsigned char *tile, int off_lo, int off_hi) {
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(tile + off_lo));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(tile + off_hi));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Byte offset, inside an LdsTile<D>, of the 8-byte piece lane `lane` passes to
// ds_read_b64_tr_b16 when reading columns [e0, e0+16) over rows [r0, r0+4).
template <int D>
__device__ __forceinline__ int tr_piece_off(int r0, int e0, int lane) {
  const int c = lane & 15;
  const int col = e0 + 4 * (c & 3);
  return LdsTile<D>::off(r0 + (c >> 2), col >> 3) + ((col & 4) << 1);
}

}  // namespace basp
