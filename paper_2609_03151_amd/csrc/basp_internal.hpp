// basp_internal.hpp -- host-side launch interfaces between the C ABI layer
// (basp_api.cpp) and the kernel translation units.  Shapes arrive here
// already validated.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/basp.h"

namespace basp {

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
  // High half of m*n written as a 64-bit product, which the device compiler
  // turns into one multiply-high; callable on the host for checking.
  __host__ __device__ __forceinline__ uint32_t div(uint32_t n) const {
    const uint32_t t1 = (uint32_t)(((uint64_t)m * n) >> 32);
    return (t1 + ((n - t1) >> s1)) >> s2;
  }
};

// Work schedule of the key-stationary backward pass (dV and dK).  A key
// tile is kKvKeys keys; the rows it needs, [k0, S), are cut at multiples of
// the chunk (kv_chunk_rows(S), T key tiles long), and a unit is one (key
// tile kt, row chunk ch) pair that writes its own partial sum.  Per
// (sequence, kv head) there are kv_units(n, T) units for n row chunks: first
// the units that start at their chunk's first row ("full"), chunk by chunk
// (chunk ch has tiles 0 .. ch*T of them); then the diagonal units (key tile
// inside its first chunk but not at its start), longest first (exactly so
// when S fills whole chunks; a partial last chunk's are shorter).  Units
// whose tile lies past S, or whose rows are empty, do nothing.  Longer chunks
// mean fewer partial sums to write and add, shorter ones more, smaller units
// to balance; a quarter of the sequence, between 2048 and 8192 rows,
// measured best.  Past S = 128K the cap grows with S so that there are at
// most 16 chunks: the partial sums take (chunks x S) rows of workspace,
// which would otherwise grow with S squared.  Host-callable for checking.
constexpr int kKvKeys = 128;
constexpr int kKvMaxChunks = 16;

__host__ __device__ inline int kv_chunk_rows(int S) {
  int rows = (S / 4) / kKvKeys * kKvKeys;
  if (rows < 2048) rows = 2048;
  int cap = ((S + kKvMaxChunks - 1) / kKvMaxChunks + kKvKeys - 1) / kKvKeys * kKvKeys;
  if (cap < 8192) cap = 8192;
  if (rows > cap) rows = cap;
  return rows;
}
__host__ __device__ inline int kv_units(int nchunks, int T) {
  return T * nchunks * (nchunks - 1) / 2 + nchunks + nchunks * (T - 1);
}
__host__ __device__ inline void kv_unit(int u, int nchunks, int T, int &kt, int &ch) {
  ch = 0;
  while (ch < nchunks && u >= ch * T + 1) {  // full units of chunk ch
    u -= ch * T + 1;
    ++ch;
  }
  if (ch < nchunks) {
    kt = u;
  } else {  // diagonal units, j-th key tile of its chunk
    ch = u % nchunks;
    kt = ch * T + u / nchunks + 1;
  }
}
// Row steps of `step_rows` at the start of a unit's rows r_lo.. that overlap
// some key of its tile [k0, k0 + kKvKeys) in a wave's 32-key block: the
// masked steps, at most ceil((k0 + kKvKeys - 1 - r_lo) / step_rows).  Every
// later step starts at or after k0 + kKvKeys - 1.
__host__ __device__ inline int kv_masked_steps(int k0, int r_lo, int steps, int step_rows) {
  const int dm = k0 + kKvKeys - 1 - r_lo;
  if (dm <= 0) return 0;
  const int n = (dm + step_rows - 1) / step_rows;
  return n < steps ? n : steps;
}

// How the attention kernels find one tensor of the share.  Row r (a token
// of the full sequence) of sequence beta lies in buffer p[r / rows], at row
// r % rows of that buffer; a row holds row_elems elements, among them the
// rank's heads from head0 on, d elements each:
//   p[r / rows] + ((beta * rows + r % rows) * row_elems + (head0 + h) * d + e)
// A head-sharded local tensor [b, S, nl, d] is the one-buffer case
// (rows = S, row_elems = nl*d, head0 = 0).  The G sequence shards
// [b, S/G, n, d] of the exchange are G buffers (rows = S/G, row_elems = n*d,
// head0 = rank*n/G), so the kernels read and write them in place.  The
// view travels as a kernel argument: 64 buffers keep the largest argument
// list (the key-stationary pass, six views) near 3.3 KB.
constexpr int kMaxViewBuffers = 64;

struct RowView {
  const void *p[kMaxViewBuffers];
  FastDiv by_rows;  // division by `rows`
  uint32_t rows, row_elems, head0;
};

RowView local_view(const void *p, int S, int nl, int d);
RowView shard_view(const void *const *shards, int G, int S, int n, int d, int rank);

// Element pointer of row r of (beta, head h) in view v, and in `left` the
// rows of that buffer from r on.  SH = false: v is known to be one buffer
// (no division).  r must be wave-uniform for the pointer to stay scalar.
template <bool SH, typename T>
__device__ __forceinline__ T *view_row(const RowView &v, int beta, uint32_t r, int h, int d,
                                       uint32_t &left) {
  uint32_t j = 0, t = r;
  if constexpr (SH) {
    j = v.by_rows.div(r);
    t = r - j * v.rows;
  }
  left = v.rows - t;
  return static_cast<T *>(const_cast<void *>(v.p[j])) +
         (((size_t)beta * v.rows + t) * v.row_elems + (size_t)(v.head0 + h) * d);
}

// Every permutation of the library is a batch of strided row copies: G*b
// blocks (member j, sequence beta) of Sg rows, each row a contiguous run of
// row_bytes.  Row t of block (j, beta) goes from
//   src_tab[j] + beta*src_beta + j*src_j + t*src_row + src_off
// to the same expression on the dst side (all in bytes).  A side that is a
// single buffer repeats its pointer in all G table entries.
//
// Two fp32 variants reduce instead of copying (gradients of a kv head that
// several members share): kAddDst adds the source row into the destination
// row; kSumSrc writes the in-order sum of `reps` source rows spaced src_rep
// bytes apart (the first taken as is, each next one added).
enum class PermMode { kCopy, kAddDst, kSumSrc };

struct PermShape {
  int b, G, Sg;
  uint64_t row_bytes;
  uint64_t src_beta, src_j, src_row, src_off;
  uint64_t dst_beta, dst_j, dst_row, dst_off;
  int vec_bytes;  // 16, 8, 4 or 2: widest access every row start allows
  PermMode mode;  // kCopy unless set; the other two need fp32 rows
  int reps;       // kSumSrc: source rows per destination row
  uint64_t src_rep;
};

hipError_t launch_permute(const void *const *src_tab, void *const *dst_tab, const PermShape &s,
                          hipStream_t stream);

// One permutation with its pointer tables, ready to launch.
struct PermCall {
  PermShape s;
  const void *src[BASP_MAX_GROUP];
  void *dst[BASP_MAX_GROUP];
};

// Up to three permutations in one launch when each has at most
// kMaxBatchBuffers members and all take the same vector width (at least 4
// bytes); otherwise one launch each.  Results are those of launch_permute.
constexpr int kMaxBatchBuffers = 16;
hipError_t launch_permute_batch(const PermCall *calls, int n, hipStream_t stream);

// The owner's send-side split of an fp32 tensor with the conversion to bf16
// fused (round to nearest even): like a kCopy PermShape, but every offset and
// the row length count elements (4 bytes read, 2 written), and vec_elems (4
// or 1) elements move together.
struct CastShape {
  int b, G, Sg;
  uint64_t row_elems;
  uint64_t src_beta, src_j, src_row, src_off;
  uint64_t dst_beta, dst_j, dst_row, dst_off;
  int vec_elems;
};

hipError_t launch_cast_bf16(const float *const *src_tab, uint16_t *const *dst_tab,
                            const CastShape &s, hipStream_t stream);

struct AttnShape {
  int b, S, Hl, Hkl, d;  // local heads
  float scale;
};

// `sharded`: the views may span several buffers (sequence shards whose row
// count is a multiple of 256, so no workgroup tile straddles two of them).
hipError_t launch_attn_fwd(const RowView &q, const RowView &k, const RowView &v,
                           const RowView &o, float *lse, const AttnShape &s, bool sharded,
                           hipStream_t stream);

// Workspace of the backward: the planes LSE * log2(e) and -D, each
// [b][Hl][Sp] fp32 with Sp = S rounded up to 64 (padding rows zero), then,
// when the key pass runs in more than one row chunk, the dV and dK partial
// sums [chunk][b][S][Hkl][d] (fp32).  Host-callable.
struct BwdChunks {
  int rows;   // rows per chunk (a multiple of kKvKeys)
  int T;      // key tiles per chunk
  int n;      // row chunks
  int units;  // work units per (sequence, kv head)
  size_t part_offset_floats;
};

__host__ __device__ inline int bwd_plane_rows(int S) { return (S + 63) / 64 * 64; }

inline BwdChunks bwd_chunks(const AttnShape &s) {
  BwdChunks ck;
  ck.rows = kv_chunk_rows(s.S);
  ck.T = ck.rows / kKvKeys;
  ck.n = (s.S + ck.rows - 1) / ck.rows;
  if (ck.n < 1) ck.n = 1;
  ck.units = kv_units(ck.n, ck.T);
  const size_t ld_floats = 2 * (size_t)s.b * s.Hl * bwd_plane_rows(s.S);
  ck.part_offset_floats = (ld_floats + 63) & ~(size_t)63;  // 256-byte aligned
  return ck;
}

inline size_t attn_bwd_workspace_bytes(const AttnShape &s) {
  const BwdChunks ck = bwd_chunks(s);
  size_t floats = ck.part_offset_floats;
  if (ck.n > 1) floats += 2 * (size_t)ck.n * s.b * s.Hkl * s.S * s.d;
  return floats * sizeof(float);
}

// Device address of the static scratch buffer of basp_attn_bwd_noalloc
// (BASP_NOALLOC_SCRATCH_BYTES) on the device of `stream` (the current device
// for the null stream), looked up once per device.  Allocates nothing.
hipError_t noalloc_scratch(hipStream_t stream, void **ptr);

// q, k, v and d_o must be one-buffer (local) views, also when `sharded`
// (then only o and the gradients are shard views).
hipError_t launch_attn_bwd(const RowView &q, const RowView &k, const RowView &v,
                           const RowView &o, const float *lse, const RowView &d_o,
                           const RowView &dq, const RowView &dk, const RowView &dv,
                           void *workspace, const AttnShape &s, bool sharded,
                           hipStream_t stream);

}  // namespace basp
