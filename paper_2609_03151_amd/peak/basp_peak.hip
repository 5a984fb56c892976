// basp_peak.hip -- two measurement kernels that give the achievable peaks the
// benchmark reports next to the published ones (a second denominator for the
// roofline fractions).  Not part of libbasp: built as libbasp_peak.so.
//
//   basp_peak_mfma_bf16  back-to-back v_mfma_f32_32x32x16_bf16 on register
//                        operands, eight independent accumulators per wave,
//                        two waves per SIMD on every CU: the matrix-core issue
//                        rate with nothing else to do.
//   basp_peak_copy       a streaming device copy, 16-byte non-temporal loads
//                        and stores, several in flight per lane: the HBM rate
//                        a plain permutation-free copy reaches.
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kAcc = 8;

__global__ __launch_bounds__(512) void mfma_peak_kernel(int iters, float *__restrict__ out) {
  const int lane = threadIdx.x & 63;
  // Operands depend on the lane so that nothing folds; values stay small.
  bf16x8 a, b;
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (float)((lane + i) & 7));
    b[i] = (__bf16)(0.001f * (float)((lane * 3 + i) & 7));
  }
  f32x16 acc[kAcc];
  for (int j = 0; j < kAcc; ++j)
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < kAcc; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
  }
  float s = 0.f;
  for (int j = 0; j < kAcc; ++j)
    for (int r = 0; r < 16; ++r) s += acc[j][r];
  out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

constexpr int kCopyThreads = 256;

// Each pass of a workgroup moves 256*U consecutive 16-byte vectors (thread t
// takes t, t + 256, ...: every load instruction of a wave is one contiguous
// 1 KiB run); the workgroups then step over the buffer in passes of
// gridDim.x*256*U vectors.  U vectors are in flight per thread.
template <int U>
__global__ __launch_bounds__(kCopyThreads) void copy_kernel(const u32x4 *__restrict__ src,
                                                            u32x4 *__restrict__ dst, size_t n16) {
  const size_t step = (size_t)gridDim.x * kCopyThreads * U;
  for (size_t b0 = (size_t)blockIdx.x * kCopyThreads * U; b0 < n16; b0 += step) {
    const size_t i0 = b0 + threadIdx.x;
    if (b0 + (size_t)kCopyThreads * U <= n16) {
      u32x4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(src + i0 + u * kCopyThreads);
#pragma unroll
      for (int u = 0; u < U; ++u) __builtin_nontemporal_store(v[u], dst + i0 + u * kCopyThreads);
    } else {
      for (int u = 0; u < U; ++u) {
        const size_t i = i0 + (size_t)u * kCopyThreads;
        if (i < n16) __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
      }
    }
  }
}

}  // namespace

extern "C" {

// FLOPs one call performs: blocks * 512 threads / 64 * iters * 8 * 32*32*16*2.
// `out` receives one float per thread (blocks * 512), keeping the work live.
int basp_peak_mfma_bf16(int blocks, int iters, float *out, void *stream) {
  if (blocks < 1 || iters < 1 || !out) return 2;
  hipLaunchKernelGGL(mfma_peak_kernel, dim3(blocks), dim3(512), 0, (hipStream_t)stream, iters,
                     out);
  return hipGetLastError() == hipSuccess ? 0 : 7;
}

// dst[0, bytes) = src[0, bytes); both 16-byte aligned, bytes a multiple of 16;
// `blocks` workgroups, `unroll` (4, 8 or 16) vectors in flight per thread.
int basp_peak_copy(const void *src, void *dst, size_t bytes, int blocks, int unroll,
                   void *stream) {
  if (!src || !dst || (bytes & 15) || ((uintptr_t)src & 15) || ((uintptr_t)dst & 15) ||
      blocks < 1 || (unroll != 4 && unroll != 8 && unroll != 16))
    return 2;
  if (bytes == 0) return 0;
  const hipStream_t st = (hipStream_t)stream;
  const u32x4 *s = (const u32x4 *)src;
  u32x4 *d = (u32x4 *)dst;
  if (unroll == 4)
    hipLaunchKernelGGL(copy_kernel<4>, dim3(blocks), dim3(kCopyThreads), 0, st, s, d, bytes / 16);
  else if (unroll == 8)
    hipLaunchKernelGGL(copy_kernel<8>, dim3(blocks), dim3(kCopyThreads), 0, st, s, d, bytes / 16);
  else
    hipLaunchKernelGGL(copy_kernel<16>, dim3(blocks), dim3(kCopyThreads), 0, st, s, d, bytes / 16);
  return hipGetLastError() == hipSuccess ? 0 : 7;
}

}  // extern "C"
