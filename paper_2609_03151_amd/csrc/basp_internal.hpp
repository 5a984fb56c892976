// basp_internal.hpp -- host-side launch interfaces between the C ABI layer
// (basp_api.cpp) and the kernel translation units.  Shapes arrive here
// already validated.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/basp.h"

namespace basp {

struct PermShape {
  int b, S, G;
  uint64_t row_bytes;        // nl*d*elem: one token's run of the rank's heads
  uint64_t shard_row_bytes;  // n*d*elem:  one token of a shard
  uint64_t head_off_bytes;   // rank*nl*d*elem
  int vec_bytes;             // 16, 8, 4 or 2: widest access every row allows
};

hipError_t launch_permute(bool is_pack, const void *const *shards, void *local,
                          const PermShape &s, hipStream_t stream);

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
