// basp_internal.hpp -- host-side launch interfaces between the C ABI layer
// (basp_api.cpp) and the kernel translation units.  Shapes arrive here
// already validated.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/basp.h"

namespace basp {

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

struct AttnShape {
  int b, S, Hl, Hkl, d;  // local heads
  float scale;
};

hipError_t launch_attn_fwd(const void *q, const void *k, const void *v, void *o,
                           float *lse, const AttnShape &s, hipStream_t stream);

size_t attn_bwd_workspace_bytes(const AttnShape &s);

hipError_t launch_attn_bwd(const void *q, const void *k, const void *v,
                           const void *o, const float *lse, const void *d_o,
                           float *dq, float *dk, float *dv, void *workspace,
                           const AttnShape &s, hipStream_t stream);

}  // namespace basp
