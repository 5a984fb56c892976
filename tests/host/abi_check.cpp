// Host build of libbasp's C ABI layer (basp_api.cpp) with every kernel launch
// replaced by a recorder, meant to run under AddressSanitizer and
// UndefinedBehaviorSanitizer.  It drives the argument checks with the misuses
// the ABI documents (each must return its status code and launch nothing),
// with extreme sizes (near INT_MAX, negative, zero), and with valid calls on
// fake aligned addresses, whose recorded launch parameters must follow the
// layouts of include/basp.h.  Prints "abi ok <cases>"; exits 1 at the first
// failure.
#include "../../paper_2609_03151_amd/csrc/basp_api.cpp"

#include <limits.h>
#include <stdio.h>

namespace basp {
static int g_launches = 0;
static PermShape g_perm;
static AttnShape g_attn;
static bool g_sharded = false;
hipError_t launch_permute(const void *const *, void *const *, const PermShape &s, hipStream_t) {
  ++g_launches;
  g_perm = s;
  return hipSuccess;
}
hipError_t launch_permute_batch(const PermCall *calls, int n, hipStream_t) {
  ++g_launches;
  if (n > 0) g_perm = calls[0].s;
  return hipSuccess;
}
hipError_t launch_cast_bf16(const float *const *, uint16_t *const *, const CastShape &s,
                            hipStream_t) {
  ++g_launches;
  if (s.vec_elems != 4 || s.row_elems != 4 * 64) return hipErrorInvalidValue;
  return hipSuccess;
}
hipError_t launch_attn_fwd(const RowView &, const RowView &, const RowView &, const RowView &,
                           float *, const AttnShape &s, bool sharded, hipStream_t) {
  ++g_launches;
  g_attn = s;
  g_sharded = sharded;
  return hipSuccess;
}
hipError_t launch_attn_bwd(const RowView &, const RowView &, const RowView &, const RowView &,
                           const float *, const RowView &, const RowView &, const RowView &,
                           const RowView &, void *, const AttnShape &s, bool sharded,
                           hipStream_t) {
  ++g_launches;
  g_attn = s;
  g_sharded = sharded;
  return hipSuccess;
}
static int g_scratch_lookups = 0;
hipError_t noalloc_scratch(hipStream_t, void **ptr) {
  ++g_scratch_lookups;
  *ptr = reinterpret_cast<void *>(0x7000000);
  return hipSuccess;
}
}  // namespace basp

// The ABI layer clears a stale launch error before launching; no runtime here.
extern "C" hipError_t hipGetLastError(void) { return hipSuccess; }

static int g_cases = 0;
#define EXPECT(expr, want)                                                             \
  do {                                                                                 \
    ++g_cases;                                                                         \
    const int before_ = basp::g_launches;                                              \
    const int got_ = (expr);                                                           \
    if (got_ != (want)) {                                                              \
      printf("FAIL line %d: %s returned %d, expected %d\n", __LINE__, #expr, got_, want); \
      return 1;                                                                        \
    }                                                                                  \
    if (got_ != BASP_OK && basp::g_launches != before_) {                              \
      printf("FAIL line %d: %s launched although it failed\n", __LINE__, #expr);       \
      return 1;                                                                        \
    }                                                                                  \
  } while (0)
#define CHECK(cond)                                          \
  do {                                                       \
    ++g_cases;                                               \
    if (!(cond)) {                                           \
      printf("FAIL line %d: %s\n", __LINE__, #cond);         \
      return 1;                                              \
    }                                                        \
  } while (0)

static void *fake(uintptr_t a) { return reinterpret_cast<void *>(a); }

int main() {
  const basp_dtype BF = BASP_BF16, F32 = BASP_F32;
  // ---- group formation (Alg. 1/2) and validation
  int g = -1, l = -1, k = -1;
  EXPECT(basp_group_of(4, 2, 3, &g, &l, &k), BASP_OK);
  CHECK(g == 1 && l == 1 && k == 2);
  EXPECT(basp_group_of(6, 4, 0, &g, &l, &k), BASP_ERR_SHAPE);
  EXPECT(basp_group_of(4, 8, 0, &g, &l, &k), BASP_ERR_DP_FALLBACK);
  EXPECT(basp_group_of(4, 2, 4, &g, &l, &k), BASP_ERR_RANK);
  EXPECT(basp_group_of(INT_MAX, 1, INT_MAX - 1, &g, &l, &k), BASP_OK);
  CHECK(g == 0 && l == INT_MAX - 1);
  EXPECT(basp_group_of(4, 2, 0, nullptr, &l, &k), BASP_ERR_NULL);
  EXPECT(basp_validate(1, 32768, 32, 8, 128, 4, 1), BASP_OK);
  EXPECT(basp_validate(1, 512, 12, 3, 64, 4, 0), BASP_ERR_SHAPE);
  EXPECT(basp_validate(1, 512, 8, 8, 72, 2, 0), BASP_ERR_UNSUPPORTED);
  EXPECT(basp_validate(INT_MAX, INT_MAX, INT_MAX, INT_MAX, 128, 1, 0), BASP_ERR_UNSUPPORTED);
  EXPECT(basp_validate(-1, 512, 8, 8, 64, 2, 0), BASP_ERR_SHAPE);
  EXPECT(basp_validate(1, 512, 8, 8, 64, 0, 0), BASP_ERR_SHAPE);
  EXPECT(basp_validate(1, 512, 8, 8, 64, 2, INT_MIN), BASP_ERR_RANK);
  for (int s = -2; s < 12; ++s) CHECK(basp_status_str(s) != nullptr);

  // ---- permutations
  void *two[2] = {fake(0x10000), fake(0x20000)};
  void *dst = fake(0x30000);
  EXPECT(basp_pack(two, dst, 1, 63, 8, 64, 2, 0, BF, nullptr), BASP_ERR_SHAPE);
  EXPECT(basp_pack(two, dst, 1, 64, 8, 64, 2, 2, BF, nullptr), BASP_ERR_RANK);
  EXPECT(basp_pack(two, dst, 1, 64, 8, 64, 2, 0, (basp_dtype)5, nullptr), BASP_ERR_UNSUPPORTED);
  EXPECT(basp_pack(two, dst, 1, 64, 8, 64, 2, 0, (basp_dtype)-1, nullptr), BASP_ERR_UNSUPPORTED);
  EXPECT(basp_pack(nullptr, dst, 1, 64, 8, 64, 2, 0, BF, nullptr), BASP_ERR_NULL);
  void *mis[2] = {fake(0x10001), fake(0x20000)};
  EXPECT(basp_pack(mis, dst, 1, 64, 8, 64, 2, 0, BF, nullptr), BASP_ERR_ALIGN);
  EXPECT(basp_pack(two, dst, 1, 1 << 22, 32, 64, 2, 0, BF, nullptr), BASP_ERR_UNSUPPORTED);
  EXPECT(basp_pack(two, dst, INT_MAX, 64, 8, 64, 2, 0, BF, nullptr), BASP_ERR_UNSUPPORTED);
  EXPECT(basp_pack(two, dst, 1, INT_MAX - 1, 8, 64, 2, 0, BF, nullptr), BASP_ERR_UNSUPPORTED);
  EXPECT(basp_pack(two, dst, 0, 64, 8, 64, 2, 0, BF, nullptr), BASP_OK);
  CHECK(basp::g_launches == 0);
  // a valid pack: [2, 64/2, 8, 64] shards -> [2, 64, 4, 64] bf16
  EXPECT(basp_pack(two, dst, 2, 64, 8, 64, 2, 1, BF, nullptr), BASP_OK);
  CHECK(basp::g_launches == 1);
  CHECK(basp::g_perm.Sg == 32 && basp::g_perm.b == 2 && basp::g_perm.G == 2);
  CHECK(basp::g_perm.row_bytes == 4 * 64 * 2);
  CHECK(basp::g_perm.src_row == 8 * 64 * 2 && basp::g_perm.src_off == 4 * 64 * 2);
  CHECK(basp::g_perm.src_beta == 32ull * 8 * 64 * 2);
  CHECK(basp::g_perm.dst_row == 4 * 64 * 2 && basp::g_perm.dst_j == 32ull * 4 * 64 * 2);
  CHECK(basp::g_perm.dst_beta == 64ull * 4 * 64 * 2);
  CHECK(basp::g_perm.vec_bytes == 16);
  EXPECT(basp_unpack(dst, two, 1, 64, 8, 64, 2, 0, F32, nullptr), BASP_OK);
  CHECK(basp::g_perm.mode == basp::PermMode::kCopy && basp::g_perm.dst_off == 0);
  void *four[4] = {fake(0x10000), fake(0x20000), fake(0x30000), fake(0x40000)};
  EXPECT(basp_unpack(dst, four, 1, 64, 2, 64, 4, 0, F32, nullptr), BASP_ERR_SHAPE);
  EXPECT(basp_unpack_add((const float *)dst, (float *const *)four, 1, 64, 2, 64, 4, 3, nullptr),
         BASP_OK);
  CHECK(basp::g_perm.mode == basp::PermMode::kAddDst && basp::g_perm.dst_off == 1 * 64 * 4);
  // odd row length: narrower accesses
  EXPECT(basp_pack(two, dst, 1, 64, 2, 3, 2, 0, BF, nullptr), BASP_OK);
  CHECK(basp::g_perm.vec_bytes == 2);
  void *big[256];
  for (int j = 0; j < 256; ++j) big[j] = fake(0x1000 * (uintptr_t)(j + 1));
  EXPECT(basp_pack(big, dst, 1, 256, 256, 8, 256, 0, BF, nullptr), BASP_ERR_UNSUPPORTED);
  EXPECT(basp_a2a_pack(dst, fake(0x50000), 1, 64, 8, 64, 2, BF, nullptr), BASP_OK);
  CHECK(basp::g_perm.dst_j == 32ull * 4 * 64 * 2);
  EXPECT(basp_a2a_unpack(dst, fake(0x50000), 1, 64, 2, 64, 4, BF, nullptr),
         BASP_ERR_UNSUPPORTED);
  EXPECT(basp_a2a_unpack(dst, fake(0x50000), 1, 64, 2, 64, 4, F32, nullptr), BASP_OK);
  CHECK(basp::g_perm.mode == basp::PermMode::kSumSrc && basp::g_perm.reps == 2 &&
        basp::g_perm.G == 2);
  EXPECT(basp_a2a_pack(dst, fake(0x50000), 32768, 64, 8, 64, 2, BF, nullptr),
         BASP_ERR_UNSUPPORTED);
  EXPECT(basp_pack_qkv(two, two, two, dst, dst, dst, 1, 64, 8, 3, 64, 2, 0, BF, nullptr),
         BASP_ERR_SHAPE);
  EXPECT(basp_pack_qkv(two, two, two, dst, dst, dst, 1, 64, 8, 2, 64, 2, 0, BF, nullptr),
         BASP_OK);
  EXPECT(basp_unpack_grads((const float *)dst, (const float *)dst, (const float *)dst,
                           (float *const *)two, (float *const *)two, (float *const *)two, 1, 64,
                           8, 2, 64, 2, -1, nullptr),
         BASP_ERR_RANK);

  // ---- attention
  void *p[10];
  for (int i = 0; i < 10; ++i) p[i] = fake(0x100000 * (uintptr_t)(i + 1));
  float *lse = (float *)p[4];
  EXPECT(basp_attn_fwd(p[0], p[1], p[2], p[3], lse, 1, 128, 8, 2, 72, 2, 0.125f, nullptr),
         BASP_ERR_UNSUPPORTED);
  EXPECT(basp_attn_fwd(p[0], p[1], p[2], p[3], lse, 1, 128, 8, 2, 128, 2, 0.f, nullptr),
         BASP_ERR_UNSUPPORTED);
  EXPECT(basp_attn_fwd(p[0], p[1], p[2], p[3], lse, 1, 128, 8, 2, 128, 2, -1.f, nullptr),
         BASP_ERR_UNSUPPORTED);
  EXPECT(basp_attn_fwd(p[0], p[1], p[2], p[3], lse, 1, 128, 8, 2, 128, 2, __builtin_nanf(""),
                       nullptr),
         BASP_ERR_UNSUPPORTED);
  EXPECT(basp_attn_fwd(p[0], p[1], p[2], p[3], lse, 1, 128, 8, 2, 128, 2, __builtin_inff(),
                       nullptr),
         BASP_ERR_UNSUPPORTED);
  EXPECT(basp_attn_fwd(p[0], p[1], p[2], p[3], lse, INT_MAX, INT_MAX - 1, 8, 2, 128, 2, 0.1f,
                       nullptr),
         BASP_ERR_UNSUPPORTED);
  EXPECT(basp_attn_fwd(p[0], p[1], p[2], p[3], lse, 1, INT_MAX, 8, 2, 128, 2, 0.1f, nullptr),
         BASP_ERR_SHAPE);
  EXPECT(basp_attn_fwd(p[0], p[1], p[2], p[3], lse, 70000, 128, 8, 2, 128, 2, 0.1f, nullptr),
         BASP_ERR_UNSUPPORTED);
  EXPECT(basp_attn_fwd(nullptr, p[1], p[2], p[3], lse, 1, 128, 8, 2, 128, 2, 0.1f, nullptr),
         BASP_ERR_NULL);
  EXPECT(basp_attn_fwd(fake(0x100008), p[1], p[2], p[3], lse, 1, 128, 8, 2, 128, 2, 0.1f,
                       nullptr),
         BASP_ERR_ALIGN);
  EXPECT(basp_attn_fwd(p[0], p[1], p[2], p[3], lse, 2, 1000, 28, 4, 128, 4, 0.1f, nullptr),
         BASP_OK);
  CHECK(basp::g_attn.b == 2 && basp::g_attn.S == 1000 && basp::g_attn.Hl == 7 &&
        basp::g_attn.Hkl == 1 && !basp::g_sharded);
  EXPECT(basp_attn_fwd(p[0], p[1], p[2], p[3], lse, 1, 512, 8, 2, 96, 4, 0.1f, nullptr),
         BASP_OK);
  CHECK(basp::g_attn.Hkl == 1);  // one kv head shared by 2 members

  const size_t need = basp_attn_bwd_workspace_bytes(1, 4096, 8, 2, 128, 2);
  CHECK(need >= 2 * 4 * 4096 * 4 + 2ull * 2 * 4096 * 128 * 4 && need % 256 == 0);
  CHECK(basp_attn_bwd_workspace_bytes(1, 4095, 8, 2, 128, 2) == 0);
  CHECK(basp_attn_bwd_workspace_bytes(1, 0, 8, 2, 128, 2) == 0);  // empty: nothing needed
  float *fq = (float *)p[6], *fk = (float *)p[7], *fv = (float *)p[8];
  EXPECT(basp_attn_bwd(p[0], p[1], p[2], p[3], lse, p[5], fq, fk, fv, p[9], need - 1, 1, 4096, 8,
                       2, 128, 2, 0.1f, nullptr),
         BASP_ERR_WORKSPACE);
  EXPECT(basp_attn_bwd(p[0], p[1], p[2], p[3], lse, p[5], fq, fk, fv, nullptr, need, 1, 4096, 8,
                       2, 128, 2, 0.1f, nullptr),
         BASP_ERR_NULL);
  EXPECT(basp_attn_bwd(p[0], p[1], p[2], p[3], lse, p[5], fq, fk, fv, p[9], need, 1, 4096, 8, 2,
                       128, 2, 0.1f, nullptr),
         BASP_OK);
  CHECK(basp::g_attn.S == 4096 && basp::g_attn.Hl == 4 && basp::g_attn.Hkl == 1);
  // the allocation-free variant: same checks, the static buffer's size as the limit
  EXPECT(basp_attn_bwd_noalloc(p[0], p[1], p[2], p[3], lse, p[5], fq, fk, fv, 1, 131072, 64, 8,
                               128, 8, 0.1f, nullptr),
         BASP_ERR_WORKSPACE);
  CHECK(basp_attn_bwd_workspace_bytes(1, 131072, 64, 8, 128, 8) > BASP_NOALLOC_SCRATCH_BYTES);
  EXPECT(basp_attn_bwd_noalloc(p[0], p[1], p[2], p[3], lse, nullptr, fq, fk, fv, 1, 4096, 8, 2,
                               128, 2, 0.1f, nullptr),
         BASP_ERR_NULL);
  EXPECT(basp_attn_bwd_noalloc(p[0], p[1], p[2], p[3], lse, p[5], (float *)fake(0x700004), fk, fv,
                               1, 4096, 8, 2, 128, 2, 0.1f, nullptr),
         BASP_ERR_ALIGN);
  EXPECT(basp_attn_bwd_noalloc(p[0], p[1], p[2], p[3], lse, p[5], fq, fk, fv, 1, 4096, 8, 2, 72,
                               2, 0.1f, nullptr),
         BASP_ERR_UNSUPPORTED);
  CHECK(basp::g_scratch_lookups == 0);
  EXPECT(basp_attn_bwd_noalloc(p[0], p[1], p[2], p[3], lse, p[5], fq, fk, fv, 1, 4096, 8, 2, 128,
                               2, 0.1f, nullptr),
         BASP_OK);
  CHECK(basp::g_scratch_lookups == 1 && basp::g_attn.S == 4096);
  EXPECT(basp_attn_bwd_noalloc(nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                               nullptr, nullptr, 0, 4096, 8, 2, 128, 2, 0.1f, nullptr),
         BASP_OK);
  CHECK(basp::g_scratch_lookups == 1);

  // ---- in place on the shard buffers
  void *tq[4], *to[4], *tk[4], *tv[4], *td[4], *tdq[4], *tdk[4], *tdv[4];
  for (int j = 0; j < 4; ++j) {
    tq[j] = fake(0x1000000 * (uintptr_t)(j + 1));
    to[j] = fake(0x1000000 * (uintptr_t)(j + 5));
    tk[j] = fake(0x1000000 * (uintptr_t)(j + 9));
    tv[j] = fake(0x1000000 * (uintptr_t)(j + 13));
    td[j] = fake(0x1000000 * (uintptr_t)(j + 17));
    tdq[j] = fake(0x1000000 * (uintptr_t)(j + 21));
    tdk[j] = fake(0x1000000 * (uintptr_t)(j + 25));
    tdv[j] = fake(0x1000000 * (uintptr_t)(j + 29));
  }
  EXPECT(basp_attn_fwd_sharded(tq, tk, tv, to, lse, 1, 1024, 8, 2, 128, 4, 4, 0.1f, nullptr),
         BASP_ERR_RANK);
  EXPECT(basp_attn_fwd_sharded(tq, tk, tv, to, lse, 1, 1536, 8, 2, 128, 4, 0, 0.1f, nullptr),
         BASP_ERR_UNSUPPORTED);
  EXPECT(basp_attn_fwd_sharded(tq, tk, tv, to, lse, 1, 4096, 8, 4, 128, 4, 3, 0.1f, nullptr),
         BASP_OK);
  CHECK(basp::g_sharded && basp::g_attn.Hl == 2 && basp::g_attn.Hkl == 1);
  const size_t need_s = basp_attn_bwd_sharded_workspace_bytes(1, 4096, 8, 4, 128, 4);
  // local copies: Q and dO (2 heads each), K and V (1 head each), bf16
  CHECK(need_s == basp_attn_bwd_workspace_bytes(1, 4096, 8, 4, 128, 4) + 2ull * 4096 * 2 * 128 * 2 +
                      2ull * 4096 * 1 * 128 * 2);
  CHECK(basp_attn_bwd_sharded_workspace_bytes(0, 4096, 8, 4, 128, 4) == 0);
  EXPECT(basp_attn_bwd_sharded(tq, tk, tv, to, lse, td, (float *const *)tdq, (float *const *)tdk,
                               (float *const *)tdv, p[9], need_s - 16, 1, 4096, 8, 4, 128, 4, 1,
                               0.1f, nullptr),
         BASP_ERR_WORKSPACE);
  EXPECT(basp_attn_bwd_sharded(tq, tk, tv, to, lse, td, (float *const *)tdq, (float *const *)tdk,
                               (float *const *)tdv, p[9], need_s, 1, 4096, 8, 4, 128, 4, 1, 0.1f,
                               nullptr),
         BASP_OK);
  // a kv head shared by two members: partial dK, dV into send blocks, accepted
  EXPECT(basp_attn_bwd_sharded(tq, tk, tv, to, lse, td, (float *const *)tdq, (float *const *)tdk,
                               (float *const *)tdv, p[9], need_s, 1, 4096, 8, 2, 128, 4, 3, 0.1f,
                               nullptr),
         BASP_OK);
  CHECK(basp::g_sharded && basp::g_attn.Hkl == 1 && basp::g_attn.Hl == 2);
  // the send-side split with the fp32 -> bf16 cast: checks, then the launch
  EXPECT(basp_a2a_pack_bf16((const float *)dst, fake(0x50001), 1, 64, 8, 64, 2, nullptr),
         BASP_ERR_ALIGN);
  EXPECT(basp_a2a_pack_bf16((const float *)dst, fake(0x50000), 1, 64, 6, 64, 4, nullptr),
         BASP_ERR_SHAPE);
  EXPECT(basp_a2a_pack_bf16((const float *)dst, fake(0x50000), 1, 64, 8, 64, 2, nullptr),
         BASP_OK);
  printf("abi ok %d\n", g_cases);
  return 0;
}
