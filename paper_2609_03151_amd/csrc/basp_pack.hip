// basp_pack.hip -- the rank-local halves of the head-parallel all-to-all
// (Sec. II-C of the paper; inside a batch-aware group, Sec. IV-C).
//
// pack:   G sequence shards [b, S/G, n, d] -> [b, S, n/G, d]
//         dst[beta][j*S/G + t][h][e] = shard_j[beta][t][rank*n/G + h][e]
// unpack: the inverse, written into the rank's head slice of each shard.
//
// For one token the rank's heads are a contiguous run of nl*d elements on
// both sides, so for each (sequence beta, shard j) either kernel is a 2-D
// copy of S/G rows: the local side is contiguous (rows j*S/G .. of sequence
// beta), the shard side strided by the shard's row length, at head offset
// rank*nl.  Workgroup L works on block (beta, j) number L % (b*G);
// each thread moves V-sized vectors (16 bytes when the row length and the
// pointers allow), U of them in flight, with non-temporal accesses: every
// byte is touched exactly once.  The only index arithmetic per vector is a
// division by the row length, done as a multiply-high.
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

// n / d for 32-bit n and a divisor d fixed per launch, by multiplication
// (Granlund and Montgomery, "Division by invariant integers using
// multiplication", 1994: the round-up multiplier with the fix-up add).
struct FastDiv {
  uint32_t m, s1, s2;
  static FastDiv make(uint32_t d) {
    uint32_t l = 0;
    while (l < 32 && (1ull << l) < d) ++l;  // ceil(log2 d)
    FastDiv f;
    f.m = (uint32_t)((((1ull << 32) * ((1ull << l) - d)) / d + 1) & 0xFFFFFFFFull);
    f.s1 = l < 1 ? l : 1;
    f.s2 = l > 1 ? l - 1 : 0;
    return f;
  }
  __device__ __forceinline__ uint32_t div(uint32_t n) const {
    const uint32_t t1 = __umulhi(m, n);
    return (t1 + ((n - t1) >> s1)) >> s2;
  }
};

// One (beta, shard) block of rows.  `rows_vecs` = S/G * row_vecs vectors on
// the local side, contiguous; shard-side row rt starts at rt * shard_row_vecs.
struct CopyGeom {
  uint32_t row_vecs;        // nl*d*elem / sizeof(V)
  FastDiv by_row;           // division by row_vecs
  uint32_t block_vecs;      // S/G * row_vecs (< 2^32, checked on the host)
  uint32_t S, Sg, G;
  uint32_t jb_count, bx_count;  // (beta, shard) blocks, and workgroups per block
  uint64_t shard_row_vecs;  // n*d*elem / sizeof(V)
  uint64_t head_off_vecs;   // rank*nl*d*elem / sizeof(V)
};

template <typename V, int U>
__global__ __launch_bounds__(256) void pack_kernel(ShardTable src, V *__restrict__ dst,
                                                   CopyGeom g) {
  const uint32_t jb = blockIdx.x % g.jb_count, bx = blockIdx.x / g.jb_count;
  const uint32_t j = jb % g.G, beta = jb / g.G;
  const V *s = static_cast<const V *>(src.p[j]) + (uint64_t)beta * g.Sg * g.shard_row_vecs +
               g.head_off_vecs;
  V *d = dst + ((uint64_t)beta * g.S + (uint64_t)j * g.Sg) * g.row_vecs;
  const uint32_t step = g.bx_count * 256u * U;
  for (uint32_t base = bx * 256u * U + threadIdx.x; base < g.block_vecs; base += step) {
    V v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = base + u * 256u;
      if (i < g.block_vecs) {
        const uint32_t rt = g.by_row.div(i);
        v[u] = nt_load(s + (uint64_t)rt * g.shard_row_vecs + (i - rt * g.row_vecs));
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = base + u * 256u;
      if (i < g.block_vecs) nt_store(v[u], d + i);
    }
  }
}

template <typename V, int U>
__global__ __launch_bounds__(256) void unpack_kernel(const V *__restrict__ src, ShardTable dst,
                                                     CopyGeom g) {
  const uint32_t jb = blockIdx.x % g.jb_count, bx = blockIdx.x / g.jb_count;
  const uint32_t j = jb % g.G, beta = jb / g.G;
  const V *s = src + ((uint64_t)beta * g.S + (uint64_t)j * g.Sg) * g.row_vecs;
  V *d = static_cast<V *>(const_cast<void *>(dst.p[j])) + (uint64_t)beta * g.Sg * g.shard_row_vecs +
         g.head_off_vecs;
  const uint32_t step = g.bx_count * 256u * U;
  for (uint32_t base = bx * 256u * U + threadIdx.x; base < g.block_vecs; base += step) {
    V v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = base + u * 256u;
      if (i < g.block_vecs) v[u] = nt_load(s + i);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = base + u * 256u;
      if (i < g.block_vecs) {
        const uint32_t rt = g.by_row.div(i);
        nt_store(v[u], d + (uint64_t)rt * g.shard_row_vecs + (i - rt * g.row_vecs));
      }
    }
  }
}

namespace {

template <typename V>
hipError_t launch_typed(bool is_pack, const void *const *shards, void *local,
                        const PermShape &s, hipStream_t stream) {
  constexpr int U = 8;
  const uint64_t vsz = sizeof(V);
  CopyGeom g;
  g.row_vecs = (uint32_t)(s.row_bytes / vsz);
  g.by_row = FastDiv::make(g.row_vecs);
  g.S = (uint32_t)s.S;
  g.Sg = (uint32_t)(s.S / s.G);
  g.G = (uint32_t)s.G;
  g.block_vecs = (uint32_t)((uint64_t)g.Sg * g.row_vecs);
  g.shard_row_vecs = s.shard_row_bytes / vsz;
  g.head_off_vecs = s.head_off_bytes / vsz;
  ShardTable t;
  for (int j = 0; j < s.G; ++j) t.p[j] = shards[j];
  const uint64_t blocks_y = (uint64_t)s.b * s.G;
  if (blocks_y == 0 || g.block_vecs == 0) return hipSuccess;
  // Enough workgroups in total to fill the GPU several times over, each
  // moving at least 256*U vectors per pass.
  uint64_t bx = ((uint64_t)g.block_vecs + 256 * U - 1) / (256 * U);
  const uint64_t want = (8192 + blocks_y - 1) / blocks_y;
  if (bx > want) bx = want;
  g.jb_count = (uint32_t)blocks_y;
  g.bx_count = (uint32_t)bx;
  // Consecutive workgroups take different (beta, shard) blocks, so the
  // shard buffers are read (or written) side by side.
  const dim3 grid((unsigned)(bx * blocks_y));
  if (is_pack)
    hipLaunchKernelGGL((pack_kernel<V, U>), grid, dim3(256), 0, stream, t, static_cast<V *>(local),
                       g);
  else
    hipLaunchKernelGGL((unpack_kernel<V, U>), grid, dim3(256), 0, stream,
                       static_cast<const V *>(local), t, g);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_permute(bool is_pack, const void *const *shards, void *local,
                          const PermShape &s, hipStream_t stream) {
  switch (s.vec_bytes) {
    case 16: return launch_typed<u32x4>(is_pack, shards, local, s, stream);
    case 8: return launch_typed<u32x2>(is_pack, shards, local, s, stream);
    case 4: return launch_typed<uint32_t>(is_pack, shards, local, s, stream);
    default: return launch_typed<uint16_t>(is_pack, shards, local, s, stream);
  }
}

}  // namespace basp
