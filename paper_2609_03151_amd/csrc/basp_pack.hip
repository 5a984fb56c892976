// basp_pack.hip -- the rank-local halves of the head-parallel all-to-all
// (Sec. II-C of the paper; inside a batch-aware group, Sec. IV-C).
//
// receive side, pack:       G sequence shards [b, S/G, n, d] -> [b, S, n/G, d]
//         dst[beta][j*S/G + t][h][e] = shard_j[beta][t][rank*n/G + h][e]
// send side, unpack:        the inverse, into the rank's head slice of each shard
// send side, a2a_pack:      own shard [b, S/G, n, d] -> [G, b, S/G, n/G, d]
//         send[j][beta][t][h][e] = own[beta][t][j*n/G + h][e]
// receive side, a2a_unpack: the inverse, every member's block into the own shard
// send side, a2a_pack_bf16: a2a_pack of an fp32 tensor, each element converted
//                           to bf16 on the way (round to nearest even)
//
// With fewer heads than members (n < G, G divisible by n) member r handles the
// single head r*n/G, shared by G/n members; gradients of such a head are
// reduced in fp32 instead of copied:
// send side, unpack_add:    dst[beta][t][h0][e] += local[beta][j*S/G + t][0][e]
// receive side, a2a_unpack: own[beta][t][h][e] = sum over the members j that
//                           share head h, in member order, of recv[j][beta][t][0][e]
//
// For one token the heads moved are a contiguous run of (n/G)*d elements on
// both sides, so each of these is, per (member j, sequence beta), a 2-D copy
// of S/G rows with a row stride on each side (PermShape).  Workgroup L works
// on block (j, beta) number L % (b*G), so all G buffers stream side by side;
// each thread moves V-sized vectors (16 bytes when every row start allows),
// U of them in flight, with non-temporal accesses: every byte is touched
// exactly once.  The only index arithmetic per vector is a division by the
// row length, done as a multiply-high.
#include "basp_device.hpp"
#include "basp_internal.hpp"

namespace basp {

struct ShardTable {
  const void *p[BASP_MAX_GROUP];
};

template <typename V>
__device__ __forceinline__ V nt_load(const V *p) {
  return __builtin_nontemporal_load(p);
}
template <typename V>
__device__ __forceinline__ void nt_store(V v, V *p) {
  __builtin_nontemporal_store(v, p);
}

// One launch's geometry in V-sized vectors.
struct CopyGeom {
  uint32_t row_vecs;               // row_bytes / sizeof(V)
  FastDiv by_row;                  // division by row_vecs
  uint32_t block_vecs;             // Sg * row_vecs (< 2^32, checked on the host)
  uint32_t G, jb_count, bx_count;  // members, (j, beta) blocks, workgroups per block
  uint32_t reps;                   // kSumSrc: source rows summed per destination row
  uint64_t src_beta, src_j, src_row, src_off, src_rep;
  uint64_t dst_beta, dst_j, dst_row, dst_off;
};

// Element-wise fp32 sum of two vectors that carry fp32 bit patterns.
__device__ __forceinline__ uint32_t fadd_bits(uint32_t a, uint32_t b) {
  return __float_as_uint(__uint_as_float(a) + __uint_as_float(b));
}
__device__ __forceinline__ uint32_t vadd(uint32_t a, uint32_t b) { return fadd_bits(a, b); }
__device__ __forceinline__ u32x2 vadd(u32x2 a, u32x2 b) {
  return u32x2{fadd_bits(a.x, b.x), fadd_bits(a.y, b.y)};
}
__device__ __forceinline__ u32x4 vadd(u32x4 a, u32x4 b) {
  return u32x4{fadd_bits(a.x, b.x), fadd_bits(a.y, b.y), fadd_bits(a.z, b.z), fadd_bits(a.w, b.w)};
}

// One pass of U vectors per thread at vector index `base` (+ u*256) of a
// block.  TAIL: some of them may lie past the block's end (only the last
// pass); a full pass has no per-vector checks, so the compiler keeps the
// loads unconditional.
template <typename V, int U, PermMode M, bool TAIL>
__device__ __forceinline__ void copy_pass(const V *s, V *d, const CopyGeom &g, uint32_t base) {
  V v[U];
  uint32_t rt[U], c[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const uint32_t i = base + u * 256u;
    rt[u] = g.by_row.div(i);
    c[u] = i - rt[u] * g.row_vecs;
    if (!TAIL || i < g.block_vecs) v[u] = nt_load(s + (uint64_t)rt[u] * g.src_row + c[u]);
  }
  if constexpr (M == PermMode::kSumSrc) {
    for (uint32_t r = 1; r < g.reps; ++r) {
      V w[U];
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (!TAIL || base + u * 256u < g.block_vecs)
          w[u] = nt_load(s + r * g.src_rep + (uint64_t)rt[u] * g.src_row + c[u]);
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (!TAIL || base + u * 256u < g.block_vecs) v[u] = vadd(v[u], w[u]);
    }
  }
  if constexpr (M == PermMode::kAddDst) {
    V w[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (!TAIL || base + u * 256u < g.block_vecs)
        w[u] = nt_load(d + (uint64_t)rt[u] * g.dst_row + c[u]);
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (!TAIL || base + u * 256u < g.block_vecs) v[u] = vadd(w[u], v[u]);
  }
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const uint32_t i = base + u * 256u;
    if (!TAIL || i < g.block_vecs) nt_store(v[u], d + (uint64_t)rt[u] * g.dst_row + c[u]);
  }
}

// Vectors [bx*256*U, ...) of one (member j, sequence beta) block, from s to
// d, in passes of bx_count*256*U; shared by the single-tensor and batched
// kernels.
template <typename V, int U, PermMode M>
__device__ __forceinline__ void copy_block(const V *s, V *d, const CopyGeom &g, uint32_t bx) {
  const uint32_t step = g.bx_count * 256u * U;
  for (uint32_t b0 = bx * 256u * U; b0 < g.block_vecs; b0 += step) {  // workgroup-uniform
    if (b0 + 256u * U <= g.block_vecs)
      copy_pass<V, U, M, false>(s, d, g, b0 + threadIdx.x);
    else
      copy_pass<V, U, M, true>(s, d, g, b0 + threadIdx.x);
  }
}

template <typename V, int U, PermMode M>
__global__ __launch_bounds__(256) void permute_kernel(ShardTable src, ShardTable dst, CopyGeom g) {
  const uint32_t jb = blockIdx.x % g.jb_count, bx = blockIdx.x / g.jb_count;
  const uint32_t j = jb % g.G, beta = jb / g.G;
  const V *s = static_cast<const V *>(src.p[j]) + beta * g.src_beta + j * g.src_j + g.src_off;
  V *d = static_cast<V *>(const_cast<void *>(dst.p[j])) + beta * g.dst_beta + j * g.dst_j +
         g.dst_off;
  copy_block<V, U, M>(s, d, g, bx);
}

// Up to kMaxBatch permutations in one launch (the Q, K, V packs of a step,
// or its three gradient unpacks): workgroups [first[k], first[k+1]) run
// permutation k with its own tables, geometry and mode, so small tensors do
// not each pay a launch and a ramp.
constexpr int kMaxBatch = 3;
struct BatchTable {
  const void *p[kMaxBatchBuffers];
};
struct BatchArgs {
  BatchTable src[kMaxBatch], dst[kMaxBatch];
  CopyGeom g[kMaxBatch];
  uint32_t first[kMaxBatch + 1];
  PermMode mode[kMaxBatch];
  int n;
};

template <typename V, int U>
__global__ __launch_bounds__(256) void permute_batch_kernel(const BatchArgs a) {
  int k = 0;
  while (k + 1 < a.n && blockIdx.x >= a.first[k + 1]) ++k;  // workgroup-uniform
  const CopyGeom &g = a.g[k];
  const uint32_t blk = blockIdx.x - a.first[k];
  const uint32_t jb = blk % g.jb_count, bx = blk / g.jb_count;
  const uint32_t j = jb % g.G, beta = jb / g.G;
  const V *s = static_cast<const V *>(a.src[k].p[j]) + beta * g.src_beta + j * g.src_j + g.src_off;
  V *d = static_cast<V *>(const_cast<void *>(a.dst[k].p[j])) + beta * g.dst_beta +
         j * g.dst_j + g.dst_off;
  if constexpr (sizeof(V) >= 4) {
    if (a.mode[k] == PermMode::kAddDst) return copy_block<V, U, PermMode::kAddDst>(s, d, g, bx);
    if (a.mode[k] == PermMode::kSumSrc) return copy_block<V, U, PermMode::kSumSrc>(s, d, g, bx);
  }
  copy_block<V, U, PermMode::kCopy>(s, d, g, bx);
}

// fp32 -> bf16 (round to nearest even, the hardware's packed conversion) of
// one vector: 4 floats -> 4 bf16, or 1 -> 1.
__device__ __forceinline__ u32x2 to_bf16(u32x4 v) {
  return u32x2{pack_bf16x2(__uint_as_float(v.x), __uint_as_float(v.y)),
               pack_bf16x2(__uint_as_float(v.z), __uint_as_float(v.w))};
}
__device__ __forceinline__ uint16_t to_bf16(uint32_t v) {
  return (uint16_t)(pack_bf16x2(__uint_as_float(v), 0.f) & 0xFFFFu);
}

// The cast variant of permute_kernel: geometry in vectors of VS (fp32 side)
// and VD (bf16 side), one to one.
template <typename VS, typename VD, int U>
__global__ __launch_bounds__(256) void cast_kernel(ShardTable src, ShardTable dst, CopyGeom g) {
  const uint32_t jb = blockIdx.x % g.jb_count, bx = blockIdx.x / g.jb_count;
  const uint32_t j = jb % g.G, beta = jb / g.G;
  const VS *s = static_cast<const VS *>(src.p[j]) + beta * g.src_beta + j * g.src_j + g.src_off;
  VD *d = static_cast<VD *>(const_cast<void *>(dst.p[j])) + beta * g.dst_beta + j * g.dst_j +
          g.dst_off;
  const uint32_t step = g.bx_count * 256u * U;
  for (uint32_t b0 = bx * 256u * U; b0 < g.block_vecs; b0 += step) {  // workgroup-uniform
    VS v[U];
    uint32_t rt[U], c[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = b0 + threadIdx.x + u * 256u;
      rt[u] = g.by_row.div(i);
      c[u] = i - rt[u] * g.row_vecs;
      if (i < g.block_vecs) v[u] = nt_load(s + (uint64_t)rt[u] * g.src_row + c[u]);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = b0 + threadIdx.x + u * 256u;
      if (i < g.block_vecs) nt_store(to_bf16(v[u]), d + (uint64_t)rt[u] * g.dst_row + c[u]);
    }
  }
}

namespace {

constexpr int kU = 8;  // vectors in flight per thread

// Geometry of one permutation in V-sized vectors, and its workgroups per
// block: enough in total to fill the GPU several times over, each moving at
// least 256*U vectors per pass.  Returns the number of (j, beta) blocks.
template <typename V>
uint64_t make_geom(const PermShape &s, CopyGeom &g) {
  constexpr int U = kU;
  const uint64_t vsz = sizeof(V);
  g.row_vecs = (uint32_t)(s.row_bytes / vsz);
  g.by_row = FastDiv::make(g.row_vecs);
  g.block_vecs = (uint32_t)((uint64_t)s.Sg * g.row_vecs);
  g.G = (uint32_t)s.G;
  g.src_beta = s.src_beta / vsz;
  g.src_j = s.src_j / vsz;
  g.src_row = s.src_row / vsz;
  g.src_off = s.src_off / vsz;
  g.src_rep = s.src_rep / vsz;
  g.reps = (uint32_t)(s.reps > 1 ? s.reps : 1);
  g.dst_beta = s.dst_beta / vsz;
  g.dst_j = s.dst_j / vsz;
  g.dst_row = s.dst_row / vsz;
  g.dst_off = s.dst_off / vsz;
  const uint64_t blocks = (uint64_t)s.b * s.G;
  g.jb_count = (uint32_t)blocks;
  g.bx_count = 0;
  if (blocks == 0 || g.block_vecs == 0) return 0;
  uint64_t bx = ((uint64_t)g.block_vecs + 256 * U - 1) / (256 * U);
  const uint64_t want = (8192 + blocks - 1) / blocks;
  if (bx > want) bx = want;
  g.bx_count = (uint32_t)bx;
  return blocks;
}

template <typename V, PermMode M>
hipError_t launch_typed(const void *const *src_tab, void *const *dst_tab, const PermShape &s,
                        hipStream_t stream) {
  CopyGeom g;
  const uint64_t blocks = make_geom<V>(s, g);
  if (blocks == 0) return hipSuccess;
  ShardTable ts, td;
  for (int j = 0; j < s.G; ++j) {
    ts.p[j] = src_tab[j];
    td.p[j] = dst_tab[j];
  }
  hipLaunchKernelGGL((permute_kernel<V, kU, M>), dim3((unsigned)(g.bx_count * blocks)), dim3(256),
                     0, stream, ts, td, g);
  return hipGetLastError();
}

template <typename V>
hipError_t launch_batch_typed(const PermCall *calls, int n, hipStream_t stream) {
  BatchArgs a{};
  uint64_t total = 0;
  for (int k = 0; k < n; ++k) {
    const uint64_t blocks = make_geom<V>(calls[k].s, a.g[k]);
    a.first[k] = (uint32_t)total;
    total += blocks * a.g[k].bx_count;
    a.mode[k] = calls[k].s.mode;
    for (int j = 0; j < calls[k].s.G; ++j) {
      a.src[k].p[j] = calls[k].src[j];
      a.dst[k].p[j] = calls[k].dst[j];
    }
  }
  a.first[n] = (uint32_t)total;
  a.n = n;
  if (total == 0) return hipSuccess;
  hipLaunchKernelGGL((permute_batch_kernel<V, kU>), dim3((unsigned)total), dim3(256), 0, stream, a);
  return hipGetLastError();
}

template <PermMode M>
hipError_t launch_reduce(const void *const *src_tab, void *const *dst_tab, const PermShape &s,
                         hipStream_t stream) {
  switch (s.vec_bytes) {
    case 16: return launch_typed<u32x4, M>(src_tab, dst_tab, s, stream);
    case 8: return launch_typed<u32x2, M>(src_tab, dst_tab, s, stream);
    default: return launch_typed<uint32_t, M>(src_tab, dst_tab, s, stream);
  }
}

template <typename VS, typename VD>
hipError_t launch_cast_typed(const float *const *src_tab, uint16_t *const *dst_tab,
                             const CastShape &s, hipStream_t stream) {
  constexpr int U = kU;
  const uint64_t ve = (uint64_t)s.vec_elems;
  CopyGeom g{};
  g.row_vecs = (uint32_t)(s.row_elems / ve);
  g.by_row = FastDiv::make(g.row_vecs);
  g.block_vecs = (uint32_t)((uint64_t)s.Sg * g.row_vecs);
  g.G = (uint32_t)s.G;
  g.reps = 1;
  g.src_beta = s.src_beta / ve, g.src_j = s.src_j / ve, g.src_row = s.src_row / ve;
  g.src_off = s.src_off / ve;
  g.dst_beta = s.dst_beta / ve, g.dst_j = s.dst_j / ve, g.dst_row = s.dst_row / ve;
  g.dst_off = s.dst_off / ve;
  const uint64_t blocks = (uint64_t)s.b * s.G;
  g.jb_count = (uint32_t)blocks;
  if (blocks == 0 || g.block_vecs == 0) return hipSuccess;
  uint64_t bx = ((uint64_t)g.block_vecs + 256 * U - 1) / (256 * U);
  const uint64_t want = (8192 + blocks - 1) / blocks;
  if (bx > want) bx = want;
  g.bx_count = (uint32_t)bx;
  ShardTable ts, td;
  for (int j = 0; j < s.G; ++j) {
    ts.p[j] = src_tab[j];
    td.p[j] = dst_tab[j];
  }
  hipLaunchKernelGGL((cast_kernel<VS, VD, U>), dim3((unsigned)(g.bx_count * blocks)), dim3(256), 0,
                     stream, ts, td, g);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_cast_bf16(const float *const *src_tab, uint16_t *const *dst_tab,
                            const CastShape &s, hipStream_t stream) {
  if (s.vec_elems == 4) return launch_cast_typed<u32x4, u32x2>(src_tab, dst_tab, s, stream);
  return launch_cast_typed<uint32_t, uint16_t>(src_tab, dst_tab, s, stream);
}

hipError_t launch_permute_batch(const PermCall *calls, int n, hipStream_t stream) {
  bool one_launch = n >= 1 && n <= kMaxBatch;
  int vec = 16;
  for (int k = 0; k < n; ++k) {
    one_launch = one_launch && calls[k].s.G <= kMaxBatchBuffers &&
                 calls[k].s.vec_bytes == calls[0].s.vec_bytes;
    vec = calls[k].s.vec_bytes < vec ? calls[k].s.vec_bytes : vec;
  }
  if (one_launch && vec >= 4) {
    switch (vec) {
      case 16: return launch_batch_typed<u32x4>(calls, n, stream);
      case 8: return launch_batch_typed<u32x2>(calls, n, stream);
      default: return launch_batch_typed<uint32_t>(calls, n, stream);
    }
  }
  for (int k = 0; k < n; ++k) {  // one launch each
    const hipError_t e = launch_permute(calls[k].src, calls[k].dst, calls[k].s, stream);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_permute(const void *const *src_tab, void *const *dst_tab, const PermShape &s,
                          hipStream_t stream) {
  if (s.mode == PermMode::kAddDst) return launch_reduce<PermMode::kAddDst>(src_tab, dst_tab, s, stream);
  if (s.mode == PermMode::kSumSrc) return launch_reduce<PermMode::kSumSrc>(src_tab, dst_tab, s, stream);
  switch (s.vec_bytes) {
    case 16: return launch_typed<u32x4, PermMode::kCopy>(src_tab, dst_tab, s, stream);
    case 8: return launch_typed<u32x2, PermMode::kCopy>(src_tab, dst_tab, s, stream);
    case 4: return launch_typed<uint32_t, PermMode::kCopy>(src_tab, dst_tab, s, stream);
    default: return launch_typed<uint16_t, PermMode::kCopy>(src_tab, dst_tab, s, stream);
  }
}

}  // namespace basp
