// basp_api.cpp -- the extern "C" surface declared in include/basp.h.
//
// Every argument check runs on the host before the first HIP call, so the
// library can be loaded and validated on a machine without a GPU.  Kernels
// are enqueued on the caller's stream; nothing here allocates, frees or
// synchronises.
#include <hip/hip_runtime.h>
#include <limits.h>
#include <math.h>
#include <stdint.h>

#include "../../include/basp.h"
#include "basp_internal.hpp"

namespace {

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// Shared shape rules of a rank's share: sizes, and the divisibility the
// head-parallel exchange needs (every group member gets S/G tokens of each
// sequence and H/G query heads, H_kv/G kv heads).
int check_share(int b, int S, int H, int H_kv, int d, int G) {
  if (b < 0 || S < 0 || H < 1 || H_kv < 1 || d < 1 || G < 1) return BASP_ERR_SHAPE;
  if (S % G != 0 || H % G != 0 || H_kv % G != 0 || H % H_kv != 0) return BASP_ERR_SHAPE;
  return BASP_OK;
}

int check_attn(int b, int S, int H, int H_kv, int d, int G, float scale) {
  int rc = check_share(b, S, H, H_kv, d, G);
  if (rc) return rc;
  if (d != 64 && d != 128) return BASP_ERR_UNSUPPORTED;
  if (!(scale > 0.f) || !isfinite(scale)) return BASP_ERR_UNSUPPORTED;
  // Row indices inside the kernels are 32-bit: b*S must fit, and one head's
  // span of a tensor (S rows of H/G heads) is addressed with 31-bit offsets.
  if ((long long)b * S >= (long long)INT_MAX) return BASP_ERR_UNSUPPORTED;
  if ((long long)S * (H / G) * d * 2 >= (1LL << 31)) return BASP_ERR_UNSUPPORTED;
  return BASP_OK;
}

int check_perm(const void *const *shards, const void *local, int b, int S, int n, int d,
               int G, int rank, int dtype, basp::PermShape *out) {
  if (b < 0 || S < 0 || n < 1 || d < 1 || G < 1) return BASP_ERR_SHAPE;
  if (S % G != 0 || n % G != 0) return BASP_ERR_SHAPE;
  if (rank < 0 || rank >= G) return BASP_ERR_RANK;
  if (dtype != BASP_BF16 && dtype != BASP_F32) return BASP_ERR_UNSUPPORTED;
  if (G > BASP_MAX_GROUP) return BASP_ERR_UNSUPPORTED;
  // The kernels index one (sequence, shard) block of S/G rows with 32-bit
  // element counts and put b*G blocks on a grid dimension.
  if ((uint64_t)(S / G) * (uint64_t)(n / G) * (uint64_t)d >= (1ull << 32)) return BASP_ERR_UNSUPPORTED;
  if ((uint64_t)b * (uint64_t)G > 65535) return BASP_ERR_UNSUPPORTED;
  out->b = b;
  out->S = S;
  out->G = G;
  // An empty problem touches no memory: its pointers are not inspected.
  if ((long long)b * S == 0) return BASP_OK;
  if (!shards || !local) return BASP_ERR_NULL;
  for (int j = 0; j < G; ++j)
    if (!shards[j]) return BASP_ERR_NULL;
  const uint64_t elem = dtype == BASP_BF16 ? 2 : 4;
  const uint64_t nl = (uint64_t)(n / G);
  out->row_bytes = nl * (uint64_t)d * elem;
  out->shard_row_bytes = (uint64_t)n * (uint64_t)d * elem;
  out->head_off_bytes = (uint64_t)rank * nl * (uint64_t)d * elem;
  if (!aligned(local, elem)) return BASP_ERR_ALIGN;
  for (int j = 0; j < G; ++j)
    if (!aligned(shards[j], elem)) return BASP_ERR_ALIGN;
  // Widest access that every row start on both sides allows.
  int vec = 16;
  while (vec > (int)elem) {
    bool ok = out->row_bytes % vec == 0 && aligned(local, vec);
    for (int j = 0; ok && j < G; ++j) ok = aligned(shards[j], vec);
    if (ok) break;
    vec >>= 1;
  }
  out->vec_bytes = vec;
  return BASP_OK;
}

int hip_status(hipError_t e) { return e == hipSuccess ? BASP_OK : BASP_ERR_HIP; }

}  // namespace

extern "C" {

const char *basp_status_str(int status) {
  switch (status) {
    case BASP_OK: return "BASP_OK";
    case BASP_ERR_NULL: return "BASP_ERR_NULL: a required pointer is NULL";
    case BASP_ERR_SHAPE:
      return "BASP_ERR_SHAPE: negative size or S, H, H_kv not divisible by G, or H by H_kv";
    case BASP_ERR_RANK: return "BASP_ERR_RANK: rank outside [0, G)";
    case BASP_ERR_UNSUPPORTED:
      return "BASP_ERR_UNSUPPORTED: head dim, dtype, group size or scale outside what the "
             "kernels handle";
    case BASP_ERR_ALIGN: return "BASP_ERR_ALIGN: pointer not aligned as documented";
    case BASP_ERR_WORKSPACE: return "BASP_ERR_WORKSPACE: workspace too small";
    case BASP_ERR_HIP: return "BASP_ERR_HIP: a HIP launch failed";
    case BASP_ERR_DP_FALLBACK:
      return "BASP_ERR_DP_FALLBACK: micro-batch larger than the world (plain data parallel)";
    default: return "BASP: unknown status";
  }
}

int basp_group_of(int world, int micro_batch, int global_rank, int *group, int *local_rank,
                  int *group_size) {
  if (!group || !local_rank || !group_size) return BASP_ERR_NULL;
  if (world < 1 || micro_batch < 1) return BASP_ERR_SHAPE;
  if (micro_batch > world) return BASP_ERR_DP_FALLBACK;
  if (world % micro_batch != 0) return BASP_ERR_SHAPE;
  if (global_rank < 0 || global_rank >= world) return BASP_ERR_RANK;
  const int K = world / micro_batch;
  *group = global_rank / K;
  *local_rank = global_rank % K;
  *group_size = K;
  return BASP_OK;
}

int basp_validate(int b, int S, int H, int H_kv, int d, int G, int rank) {
  int rc = check_share(b, S, H, H_kv, d, G);
  if (rc) return rc;
  if (rank < 0 || rank >= G) return BASP_ERR_RANK;
  if (d != 64 && d != 128) return BASP_ERR_UNSUPPORTED;
  if (G > BASP_MAX_GROUP) return BASP_ERR_UNSUPPORTED;
  return BASP_OK;
}

int basp_pack(const void *const *src_shards, void *dst, int b, int S, int n_heads, int d,
              int G, int rank, int dtype, void *stream) {
  basp::PermShape s;
  int rc = check_perm(src_shards, dst, b, S, n_heads, d, G, rank, dtype, &s);
  if (rc) return rc;
  if ((long long)b * S == 0) return BASP_OK;
  (void)hipGetLastError();
  return hip_status(basp::launch_permute(true, src_shards, dst, s, (hipStream_t)stream));
}

int basp_unpack(const void *src, void *const *dst_shards, int b, int S, int n_heads, int d,
                int G, int rank, int dtype, void *stream) {
  basp::PermShape s;
  int rc = check_perm(dst_shards, src, b, S, n_heads, d, G, rank, dtype, &s);
  if (rc) return rc;
  if ((long long)b * S == 0) return BASP_OK;
  (void)hipGetLastError();
  return hip_status(basp::launch_permute(false, dst_shards, const_cast<void *>(src), s,
                                         (hipStream_t)stream));
}

int basp_attn_fwd(const void *q, const void *k, const void *v, void *o, float *lse, int b,
                  int S, int H, int H_kv, int d, int G, float scale, void *stream) {
  int rc = check_attn(b, S, H, H_kv, d, G, scale);
  if (rc) return rc;
  if ((long long)b * S == 0) return BASP_OK;  // empty: no pointer is inspected
  if (!q || !k || !v || !o || !lse) return BASP_ERR_NULL;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16) ||
      !aligned(lse, 4))
    return BASP_ERR_ALIGN;
  basp::AttnShape s{b, S, H / G, H_kv / G, d, scale};
  (void)hipGetLastError();
  return hip_status(basp::launch_attn_fwd(q, k, v, o, lse, s, (hipStream_t)stream));
}

size_t basp_attn_bwd_workspace_bytes(int b, int S, int H, int H_kv, int d, int G) {
  if (check_share(b, S, H, H_kv, d, G) != BASP_OK) return 0;
  basp::AttnShape s{b, S, H / G, H_kv / G, d, 1.f};
  return basp::attn_bwd_workspace_bytes(s);
}

int basp_attn_bwd(const void *q, const void *k, const void *v, const void *o, const float *lse,
                  const void *d_o, float *dq, float *dk, float *dv, void *workspace,
                  size_t workspace_bytes, int b, int S, int H, int H_kv, int d, int G,
                  float scale, void *stream) {
  int rc = check_attn(b, S, H, H_kv, d, G, scale);
  if (rc) return rc;
  if ((long long)b * S == 0) return BASP_OK;  // empty: no pointer is inspected
  if (!q || !k || !v || !o || !lse || !d_o || !dq || !dk || !dv) return BASP_ERR_NULL;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16) ||
      !aligned(d_o, 16) || !aligned(dq, 16) || !aligned(dk, 16) || !aligned(dv, 16) ||
      !aligned(lse, 4))
    return BASP_ERR_ALIGN;
  basp::AttnShape s{b, S, H / G, H_kv / G, d, scale};
  const size_t need = basp::attn_bwd_workspace_bytes(s);
  if (workspace_bytes < need) return BASP_ERR_WORKSPACE;
  if (!workspace) return BASP_ERR_NULL;
  if (!aligned(workspace, 16)) return BASP_ERR_ALIGN;
  (void)hipGetLastError();
  return hip_status(
      basp::launch_attn_bwd(q, k, v, o, lse, d_o, dq, dk, dv, workspace, s, (hipStream_t)stream));
}

}  // extern "C"
