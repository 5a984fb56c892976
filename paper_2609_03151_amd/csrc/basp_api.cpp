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

#include <initializer_list>

#include "../../include/basp.h"
#include "basp_internal.hpp"

namespace {

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// Heads of an n-head tensor that one member handles: n/G when G divides n;
// with fewer heads than members (G divisible by n) the single head
// rank*n/G, which G/n members share.  0 when neither holds.
int heads_per_member(int n, int G) {
  if (n % G == 0) return n / G;
  return (n < G && G % n == 0) ? 1 : 0;
}

// Shared shape rules of a rank's share: sizes, and the divisibility the
// head-parallel exchange needs (every group member gets S/G tokens of each
// sequence and H/G query heads; H_kv/G kv heads, or one shared kv head when
// H_kv < G).
int check_share(int b, int S, int H, int H_kv, int d, int G) {
  if (b < 0 || S < 0 || H < 1 || H_kv < 1 || d < 1 || G < 1) return BASP_ERR_SHAPE;
  if (S % G != 0 || H % G != 0 || heads_per_member(H_kv, G) == 0 || H % H_kv != 0)
    return BASP_ERR_SHAPE;
  return BASP_OK;
}

basp::AttnShape attn_shape(int b, int S, int H, int H_kv, int d, int G, float scale) {
  return basp::AttnShape{b, S, H / G, heads_per_member(H_kv, G), d, scale};
}

int check_attn(int b, int S, int H, int H_kv, int d, int G, float scale) {
  int rc = check_share(b, S, H, H_kv, d, G);
  if (rc) return rc;
  if (d != 64 && d != 80 && d != 96 && d != 128) return BASP_ERR_UNSUPPORTED;
  if (!(scale > 0.f) || !isfinite(scale)) return BASP_ERR_UNSUPPORTED;
  // Row indices inside the kernels are 32-bit: b*S must fit, and one head's
  // span of a tensor (S rows of H/G heads) is addressed with 31-bit offsets.
  if ((long long)b * S >= (long long)INT_MAX) return BASP_ERR_UNSUPPORTED;
  if (b > 65535) return BASP_ERR_UNSUPPORTED;  // one grid dimension per sequence
  if ((long long)S * (H / G) * d * 2 >= (1LL << 31)) return BASP_ERR_UNSUPPORTED;
  return BASP_OK;
}

int hip_status(hipError_t e) { return e == hipSuccess ? BASP_OK : BASP_ERR_HIP; }

// Shape rules shared by every permutation.  The kernels index one (member,
// sequence) block of S/G rows with 32-bit vector counts that must stay below
// 2^31 including the loop stride, and put b*G blocks on one grid dimension.
int check_perm_shape(int b, int S, int n, int d, int G, int dtype) {
  if (b < 0 || S < 0 || n < 1 || d < 1 || G < 1) return BASP_ERR_SHAPE;
  if (S % G != 0 || heads_per_member(n, G) == 0) return BASP_ERR_SHAPE;
  if (dtype != BASP_BF16 && dtype != BASP_F32) return BASP_ERR_UNSUPPORTED;
  if (G > BASP_MAX_GROUP) return BASP_ERR_UNSUPPORTED;
  if ((uint64_t)(S / G) * (uint64_t)heads_per_member(n, G) * (uint64_t)d >= (1ull << 31))
    return BASP_ERR_UNSUPPORTED;
  if ((uint64_t)b * (uint64_t)G > 65535) return BASP_ERR_UNSUPPORTED;
  return BASP_OK;
}

// Pointers (G-entry tables, a single buffer repeated) and the widest access
// every row start on both sides allows.
int finish_perm(const void *const *src_tab, void *const *dst_tab, uint64_t elem,
                basp::PermShape *s) {
  for (int j = 0; j < s->G; ++j)
    if (!src_tab[j] || !dst_tab[j]) return BASP_ERR_NULL;
  for (int j = 0; j < s->G; ++j)
    if (!aligned(src_tab[j], elem) || !aligned(dst_tab[j], elem)) return BASP_ERR_ALIGN;
  const uint64_t q[] = {s->row_bytes, s->src_beta, s->src_j, s->src_row, s->src_off,
                        s->src_rep, s->dst_beta, s->dst_j, s->dst_row, s->dst_off};
  int vec = 16;
  while (vec > (int)elem) {
    bool ok = true;
    for (uint64_t x : q) ok = ok && x % vec == 0;
    for (int j = 0; ok && j < s->G; ++j) ok = aligned(src_tab[j], vec) && aligned(dst_tab[j], vec);
    if (ok) break;
    vec >>= 1;
  }
  s->vec_bytes = vec;
  return BASP_OK;
}

// Sequence-shard side [b, S/G, n, d] at head offset `head0`, or head-sharded
// side [b, S, nl, d] (nl = heads_per_member) with member j's tokens at rows
// j*S/G ..
void shard_side(int S, int n, int d, int G, uint64_t elem, uint64_t head0, uint64_t &beta,
                uint64_t &j, uint64_t &row, uint64_t &off) {
  beta = (uint64_t)(S / G) * n * d * elem;
  j = 0;
  row = (uint64_t)n * d * elem;
  off = head0 * d * elem;
}
void local_side(int S, int n, int d, int G, uint64_t elem, uint64_t &beta, uint64_t &j,
                uint64_t &row, uint64_t &off) {
  const uint64_t nl = (uint64_t)heads_per_member(n, G);
  beta = (uint64_t)S * nl * d * elem;
  j = (uint64_t)(S / G) * nl * d * elem;
  row = nl * d * elem;
  off = 0;
}

basp::PermShape perm_base(int b, int S, int n, int d, int G, uint64_t elem) {
  basp::PermShape s{};
  s.b = b;
  s.G = G;
  s.Sg = S / G;
  s.row_bytes = (uint64_t)heads_per_member(n, G) * d * elem;
  s.mode = basp::PermMode::kCopy;
  s.reps = 1;
  return s;
}

// Receive-side pack (to_local) or send-side unpack of the rank's head slice;
// `add` (fp32 only) adds the local rows into the shards instead.  Checks the
// arguments and fills `pc`; `*empty` is set when there is nothing to move
// (b*S == 0, no pointer inspected).
int prep_pack(bool to_local, bool add, const void *const *shards, const void *local, int b, int S,
              int n, int d, int G, int rank, int dtype, basp::PermCall *pc, bool *empty) {
  int rc = check_perm_shape(b, S, n, d, G, dtype);
  if (rc) return rc;
  if (rank < 0 || rank >= G) return BASP_ERR_RANK;
  // A head shared by several members cannot take one member's rows alone.
  if (!to_local && !add && n < G) return BASP_ERR_SHAPE;
  *empty = (long long)b * S == 0;
  if (*empty) return BASP_OK;
  if (!shards || !local) return BASP_ERR_NULL;
  const uint64_t elem = dtype == BASP_BF16 ? 2 : 4;
  basp::PermShape &s = pc->s;
  s = perm_base(b, S, n, d, G, elem);
  const uint64_t head0 = (uint64_t)rank * n / G;
  for (int j = 0; j < G; ++j) {
    if (to_local) {
      pc->src[j] = shards[j];
      pc->dst[j] = const_cast<void *>(local);
    } else {
      pc->src[j] = local;
      pc->dst[j] = const_cast<void *>(shards[j]);
    }
  }
  if (to_local) {
    shard_side(S, n, d, G, elem, head0, s.src_beta, s.src_j, s.src_row, s.src_off);
    local_side(S, n, d, G, elem, s.dst_beta, s.dst_j, s.dst_row, s.dst_off);
  } else {
    local_side(S, n, d, G, elem, s.src_beta, s.src_j, s.src_row, s.src_off);
    shard_side(S, n, d, G, elem, head0, s.dst_beta, s.dst_j, s.dst_row, s.dst_off);
    if (add) s.mode = basp::PermMode::kAddDst;
  }
  return finish_perm(pc->src, pc->dst, elem, &s);
}

int run_pack(bool to_local, bool add, const void *const *shards, const void *local, int b, int S,
             int n, int d, int G, int rank, int dtype, void *stream) {
  basp::PermCall pc;
  bool empty = false;
  const int rc = prep_pack(to_local, add, shards, local, b, S, n, d, G, rank, dtype, &pc, &empty);
  if (rc || empty) return rc;
  (void)hipGetLastError();
  return hip_status(basp::launch_permute(pc.src, pc.dst, pc.s, (hipStream_t)stream));
}

// Send-side split of the own shard (to_send) or its receive-side inverse.
int run_a2a(bool to_send, const void *src, void *dst, int b, int S, int n, int d, int G,
            int dtype, void *stream) {
  int rc = check_perm_shape(b, S, n, d, G, dtype);
  if (rc) return rc;
  const bool shared = n < G;  // one head per member, G/n members per head
  if (shared && !to_send && dtype != BASP_F32) return BASP_ERR_UNSUPPORTED;
  if ((long long)b * S == 0) return BASP_OK;
  if (!src || !dst) return BASP_ERR_NULL;
  const uint64_t elem = dtype == BASP_BF16 ? 2 : 4;
  basp::PermShape s = perm_base(b, S, n, d, G, elem);
  const uint64_t nl = (uint64_t)heads_per_member(n, G), Sg = (uint64_t)(S / G);
  const uint64_t hd = (uint64_t)d * elem;
  // own [b, S/G, n, d]
  const uint64_t own_beta = Sg * n * hd, own_row = (uint64_t)n * hd;
  // send/recv [G, b, S/G, nl, d]
  const uint64_t a2a_beta = Sg * nl * hd, a2a_j = (uint64_t)b * a2a_beta, a2a_row = nl * hd;
  const char *sp = static_cast<const char *>(src);
  char *dp = static_cast<char *>(dst);
  const void *st[BASP_MAX_GROUP];
  void *dt[BASP_MAX_GROUP];
  if (to_send) {
    // block j holds member j's heads: [j*n/G, +nl) of every own row
    s.src_beta = own_beta, s.src_j = 0, s.src_row = own_row;
    s.dst_beta = a2a_beta, s.dst_j = a2a_j, s.dst_row = a2a_row;
    for (int j = 0; j < G; ++j) {
      st[j] = sp + (uint64_t)j * n / G * hd;
      dt[j] = dp;
    }
  } else if (!shared) {
    s.src_beta = a2a_beta, s.src_j = a2a_j, s.src_row = a2a_row;
    s.dst_beta = own_beta, s.dst_j = nl * hd, s.dst_row = own_row;
    for (int j = 0; j < G; ++j) {
      st[j] = src;
      dt[j] = dst;
    }
  } else {
    // One launch block per head h: the sum of blocks h*R .. h*R+R-1.
    const int R = G / n;
    s.G = n;
    s.mode = basp::PermMode::kSumSrc;
    s.reps = R;
    s.src_rep = a2a_j;
    s.src_beta = a2a_beta, s.src_j = 0, s.src_row = a2a_row;
    s.dst_beta = own_beta, s.dst_j = 0, s.dst_row = own_row;
    for (int h = 0; h < n; ++h) {
      st[h] = sp + (uint64_t)h * R * a2a_j;
      dt[h] = dp + (uint64_t)h * hd;
    }
  }
  rc = finish_perm(st, dt, elem, &s);
  if (rc) return rc;
  (void)hipGetLastError();
  return hip_status(basp::launch_permute(st, dt, s, (hipStream_t)stream));
}

// Shape rules of the sharded (in-place) attention entry points, after
// check_attn: the shard buffers become the kernels' row views, so a view
// holds at most kMaxViewBuffers buffers, a shard's rows are a multiple of the
// 256-row workgroup tiles, and one buffer's head span is addressed with
// 31-bit offsets (fp32 gradients included).
int check_sharded(int S, int H, int H_kv, int d, int G, int rank) {
  if (rank < 0 || rank >= G) return BASP_ERR_RANK;
  if (G > basp::kMaxViewBuffers) return BASP_ERR_UNSUPPORTED;
  if ((S / G) % 256 != 0) return BASP_ERR_UNSUPPORTED;
  const int nmax = H > H_kv ? H : H_kv;
  if ((long long)(S / G) * nmax * d * 4 >= (1LL << 31)) return BASP_ERR_UNSUPPORTED;
  return BASP_OK;
}

int check_shard_table(const void *const *tab, int G) {
  if (!tab) return BASP_ERR_NULL;
  for (int j = 0; j < G; ++j)
    if (!tab[j]) return BASP_ERR_NULL;
  for (int j = 0; j < G; ++j)
    if (!aligned(tab[j], 16)) return BASP_ERR_ALIGN;
  return BASP_OK;
}

// Bytes of one local [b, S, nl, d] bf16 copy inside the in-place
// backward's workspace, rounded up to 256: nl = H/G (Q, dO) or the rank's kv
// heads (K, V).
size_t local_copy_bytes(const basp::AttnShape &s, int nl) {
  return ((size_t)s.b * s.S * nl * s.d * 2 + 255) & ~(size_t)255;
}
// The in-place backward's copies of Q, dO, K, V, then the backward's own
// workspace.
size_t sharded_bwd_copies_bytes(const basp::AttnShape &s) {
  return 2 * local_copy_bytes(s, s.Hl) + 2 * local_copy_bytes(s, s.Hkl);
}

}  // namespace

namespace basp {

RowView local_view(const void *p, int S, int nl, int d) {
  RowView v{};
  v.p[0] = p;
  v.rows = (uint32_t)(S > 0 ? S : 1);
  v.by_rows = FastDiv::make(v.rows);
  v.row_elems = (uint32_t)(nl * d);
  v.head0 = 0;
  return v;
}

RowView shard_view(const void *const *shards, int G, int S, int n, int d, int rank) {
  RowView v{};
  for (int j = 0; j < G; ++j) v.p[j] = shards[j];
  v.rows = (uint32_t)(S / G);
  v.by_rows = FastDiv::make(v.rows);
  v.row_elems = (uint32_t)(n * d);
  v.head0 = (uint32_t)((long long)rank * n / G);
  return v;
}

}  // namespace basp

extern "C" {

const char *basp_status_str(int status) {
  switch (status) {
    case BASP_OK: return "BASP_OK";
    case BASP_ERR_NULL: return "BASP_ERR_NULL: a required pointer is NULL";
    case BASP_ERR_SHAPE:
      return "BASP_ERR_SHAPE: negative size, S or H not divisible by G, H_kv neither a multiple nor a divisor of G, or H not divisible by H_kv";
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
  // The attention limits (head dims, 32-bit row indices), then the rank, then
  // the permutation limits of the share's Q (n = H) and K, V (n = H_kv).
  int rc = check_attn(b, S, H, H_kv, d, G, 1.f);
  if (rc) return rc;
  if (rank < 0 || rank >= G) return BASP_ERR_RANK;
  rc = check_perm_shape(b, S, H, d, G, BASP_BF16);
  if (!rc) rc = check_perm_shape(b, S, H_kv, d, G, BASP_BF16);
  return rc;
}

int basp_pack(const void *const *src_shards, void *dst, int b, int S, int n_heads, int d,
              int G, int rank, basp_dtype dtype, void *stream) {
  return run_pack(true, false, src_shards, dst, b, S, n_heads, d, G, rank, dtype, stream);
}

int basp_unpack(const void *src, void *const *dst_shards, int b, int S, int n_heads, int d,
                int G, int rank, basp_dtype dtype, void *stream) {
  return run_pack(false, false, const_cast<const void *const *>(dst_shards), src, b, S, n_heads, d, G,
                  rank, dtype, stream);
}

int basp_pack_qkv(const void *const *q_shards, const void *const *k_shards,
                  const void *const *v_shards, void *q, void *k, void *v, int b, int S, int H,
                  int H_kv, int d, int G, int rank, basp_dtype dtype, void *stream) {
  basp::PermCall pc[3];
  bool empty = false;
  int rc = prep_pack(true, false, q_shards, q, b, S, H, d, G, rank, dtype, &pc[0], &empty);
  if (!rc) rc = prep_pack(true, false, k_shards, k, b, S, H_kv, d, G, rank, dtype, &pc[1], &empty);
  if (!rc) rc = prep_pack(true, false, v_shards, v, b, S, H_kv, d, G, rank, dtype, &pc[2], &empty);
  if (rc || empty) return rc;
  (void)hipGetLastError();
  return hip_status(basp::launch_permute_batch(pc, 3, (hipStream_t)stream));
}

int basp_unpack_grads(const float *dq, const float *dk, const float *dv, float *const *dq_shards,
                      float *const *dk_shards, float *const *dv_shards, int b, int S, int H,
                      int H_kv, int d, int G, int rank, void *stream) {
  using Tab = const void *const *;
  const bool add_kv = H_kv < G;  // a shared kv head: each member adds its part
  basp::PermCall pc[3];
  bool empty = false;
  int rc = prep_pack(false, false, (Tab)dq_shards, dq, b, S, H, d, G, rank, BASP_F32, &pc[0],
                     &empty);
  if (!rc)
    rc = prep_pack(false, add_kv, (Tab)dk_shards, dk, b, S, H_kv, d, G, rank, BASP_F32, &pc[1],
                   &empty);
  if (!rc)
    rc = prep_pack(false, add_kv, (Tab)dv_shards, dv, b, S, H_kv, d, G, rank, BASP_F32, &pc[2],
                   &empty);
  if (rc || empty) return rc;
  (void)hipGetLastError();
  return hip_status(basp::launch_permute_batch(pc, 3, (hipStream_t)stream));
}

int basp_unpack_add(const float *src, float *const *dst_shards, int b, int S, int n_heads, int d,
                    int G, int rank, void *stream) {
  return run_pack(false, true, reinterpret_cast<const void *const *>(dst_shards), src, b, S,
                  n_heads, d, G, rank, BASP_F32, stream);
}

int basp_a2a_pack(const void *own, void *send, int b, int S, int n_heads, int d, int G,
                  basp_dtype dtype, void *stream) {
  return run_a2a(true, own, send, b, S, n_heads, d, G, dtype, stream);
}

int basp_a2a_unpack(const void *recv, void *own, int b, int S, int n_heads, int d, int G,
                    basp_dtype dtype, void *stream) {
  return run_a2a(false, recv, own, b, S, n_heads, d, G, dtype, stream);
}

int basp_a2a_pack_bf16(const float *own, void *send, int b, int S, int n_heads, int d, int G,
                       void *stream) {
  int rc = check_perm_shape(b, S, n_heads, d, G, BASP_F32);
  if (rc) return rc;
  if ((long long)b * S == 0) return BASP_OK;  // empty: no pointer is inspected
  if (!own || !send) return BASP_ERR_NULL;
  if (!aligned(own, 4) || !aligned(send, 2)) return BASP_ERR_ALIGN;
  const int n = n_heads;
  const uint64_t nl = (uint64_t)heads_per_member(n, G), Sg = (uint64_t)(S / G);
  basp::CastShape c{};
  c.b = b, c.G = G, c.Sg = (int)Sg;
  c.row_elems = nl * d;
  // own [b, S/G, n, d] -> send [G, b, S/G, nl, d]; block j from head j*n/G on
  c.src_beta = Sg * n * d, c.src_j = 0, c.src_row = (uint64_t)n * d, c.src_off = 0;
  c.dst_beta = Sg * nl * d, c.dst_j = b * Sg * nl * d, c.dst_row = nl * d, c.dst_off = 0;
  const float *st[BASP_MAX_GROUP];
  uint16_t *dt[BASP_MAX_GROUP];
  bool vec4 = aligned(own, 16) && aligned(send, 8) && c.row_elems % 4 == 0 && c.src_row % 4 == 0;
  for (int j = 0; j < G; ++j) {
    const uint64_t h0 = (uint64_t)j * n / G * d;  // first element of member j's heads
    st[j] = own + h0;
    dt[j] = static_cast<uint16_t *>(send);
    vec4 = vec4 && h0 % 4 == 0;
  }
  c.vec_elems = vec4 ? 4 : 1;
  (void)hipGetLastError();
  return hip_status(basp::launch_cast_bf16(st, dt, c, (hipStream_t)stream));
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
  basp::AttnShape s = attn_shape(b, S, H, H_kv, d, G, scale);
  const basp::RowView qv = basp::local_view(q, S, s.Hl, d), kv = basp::local_view(k, S, s.Hkl, d),
                      vv = basp::local_view(v, S, s.Hkl, d), ov = basp::local_view(o, S, s.Hl, d);
  (void)hipGetLastError();
  return hip_status(basp::launch_attn_fwd(qv, kv, vv, ov, lse, s, false, (hipStream_t)stream));
}

int basp_attn_fwd_sharded(const void *const *q_shards, const void *const *k_shards,
                          const void *const *v_shards, void *const *o_shards, float *lse, int b,
                          int S, int H, int H_kv, int d, int G, int rank, float scale,
                          void *stream) {
  int rc = check_attn(b, S, H, H_kv, d, G, scale);
  if (rc) return rc;
  rc = check_sharded(S, H, H_kv, d, G, rank);
  if (rc) return rc;
  if ((long long)b * S == 0) return BASP_OK;  // empty: no pointer is inspected
  for (const void *const *t : {q_shards, k_shards, v_shards, (const void *const *)o_shards})
    if ((rc = check_shard_table(t, G))) return rc;
  if (!lse) return BASP_ERR_NULL;
  if (!aligned(lse, 4)) return BASP_ERR_ALIGN;
  basp::AttnShape s = attn_shape(b, S, H, H_kv, d, G, scale);
  const basp::RowView qv = basp::shard_view(q_shards, G, S, H, d, rank),
                      kv = basp::shard_view(k_shards, G, S, H_kv, d, rank),
                      vv = basp::shard_view(v_shards, G, S, H_kv, d, rank),
                      ov = basp::shard_view(o_shards, G, S, H, d, rank);
  (void)hipGetLastError();
  return hip_status(basp::launch_attn_fwd(qv, kv, vv, ov, lse, s, true, (hipStream_t)stream));
}

size_t basp_attn_bwd_workspace_bytes(int b, int S, int H, int H_kv, int d, int G) {
  if (check_share(b, S, H, H_kv, d, G) != BASP_OK) return 0;
  basp::AttnShape s = attn_shape(b, S, H, H_kv, d, G, 1.f);
  return basp::attn_bwd_workspace_bytes(s);
}

size_t basp_attn_bwd_sharded_workspace_bytes(int b, int S, int H, int H_kv, int d, int G) {
  if (check_share(b, S, H, H_kv, d, G) != BASP_OK) return 0;
  basp::AttnShape s = attn_shape(b, S, H, H_kv, d, G, 1.f);
  if ((long long)b * S == 0) return 0;
  return sharded_bwd_copies_bytes(s) + basp::attn_bwd_workspace_bytes(s);
}

}  // extern "C"

namespace {

// Checks of the local backward's tensors; *empty when there is nothing to do.
int check_bwd_local(const void *q, const void *k, const void *v, const void *o, const float *lse,
                    const void *d_o, float *dq, float *dk, float *dv, int b, int S, int H,
                    int H_kv, int d, int G, float scale, bool *empty) {
  int rc = check_attn(b, S, H, H_kv, d, G, scale);
  if (rc) return rc;
  *empty = (long long)b * S == 0;
  if (*empty) return BASP_OK;  // empty: no pointer is inspected
  if (!q || !k || !v || !o || !lse || !d_o || !dq || !dk || !dv) return BASP_ERR_NULL;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16) ||
      !aligned(d_o, 16) || !aligned(dq, 16) || !aligned(dk, 16) || !aligned(dv, 16) ||
      !aligned(lse, 4))
    return BASP_ERR_ALIGN;
  return BASP_OK;
}

int launch_bwd_local(const void *q, const void *k, const void *v, const void *o, const float *lse,
                     const void *d_o, float *dq, float *dk, float *dv, void *workspace,
                     const basp::AttnShape &s, void *stream) {
  using basp::local_view;
  const int S = s.S, d = s.d;
  const basp::RowView qv = local_view(q, S, s.Hl, d), kv = local_view(k, S, s.Hkl, d),
                      vv = local_view(v, S, s.Hkl, d), ov = local_view(o, S, s.Hl, d),
                      dov = local_view(d_o, S, s.Hl, d), dqv = local_view(dq, S, s.Hl, d),
                      dkv = local_view(dk, S, s.Hkl, d), dvv = local_view(dv, S, s.Hkl, d);
  (void)hipGetLastError();
  return hip_status(basp::launch_attn_bwd(qv, kv, vv, ov, lse, dov, dqv, dkv, dvv, workspace, s,
                                          false, (hipStream_t)stream));
}

}  // namespace

extern "C" {

int basp_attn_bwd(const void *q, const void *k, const void *v, const void *o, const float *lse,
                  const void *d_o, float *dq, float *dk, float *dv, void *workspace,
                  size_t workspace_bytes, int b, int S, int H, int H_kv, int d, int G,
                  float scale, void *stream) {
  bool empty = false;
  int rc = check_bwd_local(q, k, v, o, lse, d_o, dq, dk, dv, b, S, H, H_kv, d, G, scale, &empty);
  if (rc || empty) return rc;
  basp::AttnShape s = attn_shape(b, S, H, H_kv, d, G, scale);
  const size_t need = basp::attn_bwd_workspace_bytes(s);
  if (workspace_bytes < need) return BASP_ERR_WORKSPACE;
  if (!workspace) return BASP_ERR_NULL;
  if (!aligned(workspace, 16)) return BASP_ERR_ALIGN;
  return launch_bwd_local(q, k, v, o, lse, d_o, dq, dk, dv, workspace, s, stream);
}

int basp_attn_bwd_noalloc(const void *q, const void *k, const void *v, const void *o,
                          const float *lse, const void *d_o, float *dq, float *dk, float *dv,
                          int b, int S, int H, int H_kv, int d, int G, float scale,
                          void *stream) {
  bool empty = false;
  int rc = check_bwd_local(q, k, v, o, lse, d_o, dq, dk, dv, b, S, H, H_kv, d, G, scale, &empty);
  if (rc || empty) return rc;
  basp::AttnShape s = attn_shape(b, S, H, H_kv, d, G, scale);
  if (basp::attn_bwd_workspace_bytes(s) > BASP_NOALLOC_SCRATCH_BYTES) return BASP_ERR_WORKSPACE;
  void *scratch = nullptr;
  if (basp::noalloc_scratch((hipStream_t)stream, &scratch) != hipSuccess) return BASP_ERR_HIP;
  return launch_bwd_local(q, k, v, o, lse, d_o, dq, dk, dv, scratch, s, stream);
}

int basp_attn_bwd_sharded(const void *const *q_shards, const void *const *k_shards,
                          const void *const *v_shards, const void *const *o_shards,
                          const float *lse, const void *const *do_shards,
                          float *const *dq_shards, float *const *dk_shards,
                          float *const *dv_shards, void *workspace, size_t workspace_bytes,
                          int b, int S, int H, int H_kv, int d, int G, int rank, float scale,
                          void *stream) {
  int rc = check_attn(b, S, H, H_kv, d, G, scale);
  if (rc) return rc;
  rc = check_sharded(S, H, H_kv, d, G, rank);
  if (rc) return rc;
  // A kv head shared by several members gets a partial gradient from each:
  // dK and dV then go to G send blocks [b, S/G, 1, d], one per destination
  // member, whose receiver sums them (basp_a2a_unpack), instead of the head
  // slices of the shard buffers, where the members would overwrite one
  // another.
  const bool shared_kv = H_kv < G;
  if ((long long)b * S == 0) return BASP_OK;  // empty: no pointer is inspected
  using Tab = const void *const *;
  for (Tab t : {q_shards, k_shards, v_shards, o_shards, do_shards, (Tab)dq_shards,
                (Tab)dk_shards, (Tab)dv_shards})
    if ((rc = check_shard_table(t, G))) return rc;
  if (!lse) return BASP_ERR_NULL;
  if (!aligned(lse, 4)) return BASP_ERR_ALIGN;
  basp::AttnShape s = attn_shape(b, S, H, H_kv, d, G, scale);
  const size_t copies = sharded_bwd_copies_bytes(s);
  const size_t need = copies + basp::attn_bwd_workspace_bytes(s);
  if (workspace_bytes < need) return BASP_ERR_WORKSPACE;
  if (!workspace) return BASP_ERR_NULL;
  if (!aligned(workspace, 16)) return BASP_ERR_ALIGN;
  // Q and dO rows are streamed once per key tile by the key-stationary pass,
  // K and V rows once per row tile by the dQ pass; read from the shards,
  // rows sit a whole shard row (all heads) apart and stream measurably
  // slower than from a local copy.  So the rank's heads of Q, dO, K and V
  // are first packed into the workspace (two launches), and the kernels read
  // those copies; O is read and the gradients written in place.
  char *ws = static_cast<char *>(workspace);
  const size_t cq = local_copy_bytes(s, s.Hl), ck = local_copy_bytes(s, s.Hkl);
  void *q_loc = ws, *do_loc = ws + cq, *k_loc = ws + 2 * cq, *v_loc = ws + 2 * cq + ck;
  basp::PermCall pc[4];
  bool empty = false;
  rc = prep_pack(true, false, q_shards, q_loc, b, S, H, d, G, rank, BASP_BF16, &pc[0], &empty);
  if (!rc) rc = prep_pack(true, false, do_shards, do_loc, b, S, H, d, G, rank, BASP_BF16, &pc[1],
                          &empty);
  if (!rc) rc = prep_pack(true, false, k_shards, k_loc, b, S, H_kv, d, G, rank, BASP_BF16, &pc[2],
                          &empty);
  if (!rc) rc = prep_pack(true, false, v_shards, v_loc, b, S, H_kv, d, G, rank, BASP_BF16, &pc[3],
                          &empty);
  if (rc) return rc;
  (void)hipGetLastError();
  rc = hip_status(basp::launch_permute_batch(pc, 2, (hipStream_t)stream));
  if (!rc) rc = hip_status(basp::launch_permute_batch(pc + 2, 2, (hipStream_t)stream));
  if (rc) return rc;
  using basp::shard_view;
  const basp::RowView qv = basp::local_view(q_loc, S, s.Hl, d),
                      kv = basp::local_view(k_loc, S, s.Hkl, d),
                      vv = basp::local_view(v_loc, S, s.Hkl, d),
                      ov = shard_view(o_shards, G, S, H, d, rank),
                      dov = basp::local_view(do_loc, S, s.Hl, d),
                      dqv = shard_view((Tab)dq_shards, G, S, H, d, rank),
                      dkv = shared_kv ? shard_view((Tab)dk_shards, G, S, 1, d, 0)
                                      : shard_view((Tab)dk_shards, G, S, H_kv, d, rank),
                      dvv = shared_kv ? shard_view((Tab)dv_shards, G, S, 1, d, 0)
                                      : shard_view((Tab)dv_shards, G, S, H_kv, d, rank);
  (void)hipGetLastError();
  return hip_status(basp::launch_attn_bwd(qv, kv, vv, ov, lse, dov, dqv, dkv, dvv,
                                          ws + copies, s, true, (hipStream_t)stream));
}

}  // extern "C"
