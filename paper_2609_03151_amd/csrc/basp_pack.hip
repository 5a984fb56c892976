// basp_pack.hip -- the rank-local halves of the head-parallel all-to-all
// (Sec. II-C of the paper; inside a batch-aware group, Sec. IV-C).
//
// pack:   G sequence shards [b, S/G, n, d] -> [b, S, n/G, d]
//         dst[beta][j*S/G + t][h][e] = shard_j[beta][t][rank*n/G + h][e]
// unpack: the inverse, written into the rank's head slice of each shard.
//
// For one token the rank's heads are a contiguous run of nl*d elements on
// both sides, so either kernel is a batch of row copies: row r of the local
// tensor (r = beta*S + s, s = j*S/G + t) <-> row (beta*S/G + t) of shard j,
// at head offset rank*nl.  Each thread moves V-sized vectors (16 bytes when
// the row length and the pointers allow), U of them in flight, with
// non-temporal accesses: every byte is touched exactly once.
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

// Row mapping shared by both directions.  `vec` indexes V-vectors of the
// local tensor; returns the shard index and the vector offset inside it.
struct RowMap {
  uint32_t row_vecs;   // nl*d*elem / sizeof(V)
  uint32_t S, Sg;
  uint64_t shard_row_vecs;  // n*d*elem / sizeof(V)
  uint64_t head_off_vecs;   // rank*nl*d*elem / sizeof(V)

  __device__ __forceinline__ void map(uint64_t vec, uint32_t &j,
                                      uint64_t &shard_off) const {
    uint64_t r = vec / row_vecs;
    uint32_t c = (uint32_t)(vec - r * row_vecs);
    uint64_t beta = r / S;
    uint32_t s = (uint32_t)(r - beta * S);
    j = s / Sg;
    uint32_t t = s - j * Sg;
    shard_off = (beta * Sg + t) * shard_row_vecs + head_off_vecs + c;
  }
};

template <typename V, int U>
__global__ __launch_bounds__(256) void pack_kernel(ShardTable src, V *__restrict__ dst,
                                                   uint64_t total, RowMap m) {
  const uint64_t stride = (uint64_t)gridDim.x * 256u;
  for (uint64_t base = (uint64_t)blockIdx.x * 256u + threadIdx.x; base < total;
       base += stride * U) {
    V v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      uint64_t idx = base + u * stride;
      if (idx < total) {
        uint32_t j;
        uint64_t off;
        m.map(idx, j, off);
        v[u] = nt_load(static_cast<const V *>(src.p[j]) + off);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      uint64_t idx = base + u * stride;
      if (idx < total) nt_store(v[u], dst + idx);
    }
  }
}

template <typename V, int U>
__global__ __launch_bounds__(256) void unpack_kernel(const V *__restrict__ src, ShardTable dst,
                                                     uint64_t total, RowMap m) {
  const uint64_t stride = (uint64_t)gridDim.x * 256u;
  for (uint64_t base = (uint64_t)blockIdx.x * 256u + threadIdx.x; base < total;
       base += stride * U) {
    V v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      uint64_t idx = base + u * stride;
      if (idx < total) v[u] = nt_load(src + idx);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      uint64_t idx = base + u * stride;
      if (idx < total) {
        uint32_t j;
        uint64_t off;
        m.map(idx, j, off);
        nt_store(v[u], static_cast<V *>(const_cast<void *>(dst.p[j])) + off);
      }
    }
  }
}

namespace {

template <typename V>
hipError_t launch_typed(bool is_pack, const void *const *shards, void *local,
                        const PermShape &s, hipStream_t stream) {
  constexpr int U = 4;
  const uint64_t vsz = sizeof(V);
  RowMap m;
  m.row_vecs = (uint32_t)(s.row_bytes / vsz);
  m.S = (uint32_t)s.S;
  m.Sg = (uint32_t)(s.S / s.G);
  m.shard_row_vecs = s.shard_row_bytes / vsz;
  m.head_off_vecs = s.head_off_bytes / vsz;
  const uint64_t total = (uint64_t)s.b * (uint64_t)s.S * m.row_vecs;
  ShardTable t;
  for (int j = 0; j < s.G; ++j) t.p[j] = shards[j];
  uint64_t blocks = (total + 256 * U - 1) / (256 * U);
  if (blocks > 32768) blocks = 32768;
  if (blocks == 0) return hipSuccess;
  if (is_pack)
    hipLaunchKernelGGL((pack_kernel<V, U>), dim3((unsigned)blocks), dim3(256), 0, stream,
                       t, static_cast<V *>(local), total, m);
  else
    hipLaunchKernelGGL((unpack_kernel<V, U>), dim3((unsigned)blocks), dim3(256), 0, stream,
                       static_cast<const V *>(local), t, total, m);
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
