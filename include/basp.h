/*
 * basp.h -- C ABI of libbasp: one GPU's share of batch-aware Ulysses
 * sequence-parallel attention (BASP, "Batch-Aware Sequence Parallelism for
 * LLM Training"), hand-written HIP for gfx950 (MI355X).
 *
 * A BASP rank belongs to a group of G = N / B GPUs (Sec. IV-A, Alg. 1); the
 * group holds b sequences, each cut into G contiguous token chunks, one per
 * member (Alg. 2, Sec. IV-B).  Around attention the group runs a G-way
 * all-to-all that turns sequence shards into head shards and back
 * (Sec. II-C, Sec. IV-C).  This library computes everything one rank does
 * around that exchange, on its own GPU:
 *
 *   basp_pack      G received sequence shards -> head-sharded full sequence
 *   basp_attn_fwd  causal GQA attention on the rank's H/G query heads
 *   basp_attn_bwd  its backward (dQ, dK, dV in fp32)
 *   basp_unpack    head-sharded result -> the rank's head slice of G shards
 *   basp_unpack_add  the same for fp32 gradients, added into the shards
 *   basp_pack_qkv / basp_unpack_grads   a step's three packs, or its three
 *                  gradient unpacks, in one launch
 *   basp_attn_fwd_sharded / basp_attn_bwd_sharded   attention straight on
 *                  the shard buffers of the exchange (no pack/unpack pass)
 *   basp_a2a_pack / basp_a2a_unpack   the owner's side of the same exchanges:
 *                  own shard <-> one contiguous block per member
 *   basp_a2a_pack_bf16  the send side for an fp32 tensor, cast to bf16
 *   basp_attn_bwd_noalloc  the backward with a static device workspace
 *
 * The exchange itself (RCCL) is not part of this library.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Shapes (row-major, innermost last; "n" is the global head count of the
 * tensor at hand: H for Q, O, dO, dQ and H_kv for K, V, dK, dV):
 *   sequence shard j      [b, S/G, n,  d]   tokens [j*S/G, (j+1)*S/G)
 *   head-sharded local    [b, S,   nl, d]   heads  [rank*n/G, rank*n/G + nl)
 *   LSE                   [b, H/G, S]       fp32, natural logarithm
 * where nl = n/G when G divides n.  A GQA model may have fewer kv heads
 * than the group has members (Sec. II-A; e.g. 8 kv heads and G = 16): when
 * n < G and G is a multiple of n, nl = 1 and member rank takes the single
 * head rank*n/G (integer division), which the G/n members
 * [h*G/n, (h+1)*G/n) share.  Their gradients of that head are partial sums
 * that must be added, not copied: basp_unpack_add and basp_a2a_unpack do
 * that in fp32; basp_unpack refuses such a tensor.
 * GQA: local query head h attends with local kv head h / (H/H_kv) (with one
 * shared kv head, every local query head uses it).
 * Attention is causal (key j is visible to query i iff j <= i, top-left
 * aligned, S queries and S keys), softmax scale is the caller's `scale`
 * (1/sqrt(d) for the usual scaled dot product of Sec. II-A).
 *
 * Memory and streams: every pointer is a device pointer owned by the caller
 * (the shard pointer arrays themselves are host arrays of G device
 * pointers).  The library never allocates, frees or synchronises; work is
 * enqueued on `stream` (a hipStream_t passed as void*, NULL = null stream)
 * and the call returns before it finishes.  Outputs must not alias inputs.
 * Functions are thread-safe and keep no state between calls.
 *
 * Errors: every host-detectable misuse is rejected with a status code
 * before any HIP call is made (the library can be loaded and validated on a
 * host without a GPU).  Launch failures return BASP_ERR_HIP; faults inside a
 * kernel surface at the caller's next synchronisation.  An empty problem
 * (b == 0 or S == 0) is valid, enqueues nothing and inspects no pointer
 * (empty tensors may have NULL data).
 */
#ifndef BASP_H
#define BASP_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum basp_status {
  BASP_OK = 0,
  BASP_ERR_NULL = 1,        /* a required pointer is NULL                    */
  BASP_ERR_SHAPE = 2,       /* negative size, S%G or H%G != 0, H_kv neither a
                               multiple nor a divisor of G, or H%H_kv != 0   */
  BASP_ERR_RANK = 3,        /* rank outside [0, G)                           */
  BASP_ERR_UNSUPPORTED = 4, /* d, dtype, G or size outside what the kernels handle */
  BASP_ERR_ALIGN = 5,       /* pointer not aligned as documented             */
  BASP_ERR_WORKSPACE = 6,   /* workspace smaller than the query reports      */
  BASP_ERR_HIP = 7,         /* a HIP launch failed                           */
  BASP_ERR_DP_FALLBACK = 8  /* micro-batch larger than the world (plain DP)  */
} basp_status;

/* Element type of a permuted tensor.  Values other than the two listed are
 * rejected with BASP_ERR_UNSUPPORTED (the last two enumerators only make the
 * type span every int, so that any int a caller passes is representable). */
typedef enum basp_dtype {
  BASP_BF16 = 0,
  BASP_F32 = 1,
  BASP_DTYPE_INT_MAX_ = 0x7fffffff,
  BASP_DTYPE_INT_MIN_ = -0x7fffffff - 1
} basp_dtype;

/* Largest group size the permutation kernels accept. */
#define BASP_MAX_GROUP 128

/* Human-readable name of a status code (static string, never NULL).  The
 * codes report, before any device work, the conditions the method requires
 * of its sizes: the group-formation assert N mod B = 0 of Alg. 1 and the
 * equal token chunks L/K of Alg. 2 are BASP_ERR_SHAPE, B > N (Sec. IV-A's
 * fall-back to data parallelism) is BASP_ERR_DP_FALLBACK. */
const char *basp_status_str(int status);

/* Batch-aware group formation (Alg. 1) and rank placement (Alg. 2):
 * world N GPUs, micro-batch B; K = N/B, groups of K contiguous ranks,
 * group = floor(rank/K), local_rank = rank mod K.  Host only.
 * Errors: SHAPE (N or B < 1, N % B != 0), DP_FALLBACK (B > N),
 * RANK (global_rank outside [0, N)), NULL. */
int basp_group_of(int world, int micro_batch, int global_rank, int *group,
                  int *local_rank, int *group_size);

/* Check a share's parameters (b, S, H, H_kv, d, G, rank) without touching
 * the GPU: the sequence splits into G equal contiguous chunks (Alg. 2,
 * S % G == 0), the query heads into G equal blocks (Sec. II-C head split,
 * H % G == 0), the kv heads into G blocks or G/H_kv members per kv head
 * (Sec. II-A GQA), H % H_kv == 0, and 0 <= rank < G.  Returns BASP_OK or the
 * code the other entry points would give for the same shape (UNSUPPORTED
 * when d is not 64, 80, 96 or 128). */
int basp_validate(int b, int S, int H, int H_kv, int d, int G, int rank);

/* Receive side of the head-parallel all-to-all (Sec. II-C, Sec. IV-C):
 *   dst[beta][j*S/G + t][h][e] = src_shards[j][beta][t][rank*n/G + h][e]
 * src_shards: host array of G device pointers, each [b, S/G, n, d];
 * dst: device [b, S, nl, d] (nl as above; a shared head is copied to each
 * of its members).  dtype selects 2-byte (BASP_BF16) or 4-byte (BASP_F32)
 * elements; values are copied bit for bit.
 * Alignment: every pointer aligned to the element size.
 * Errors: NULL, SHAPE (S % G, or n neither a multiple nor a divisor of G),
 * RANK, UNSUPPORTED (dtype, G > BASP_MAX_GROUP, (S/G)*nl*d >= 2^31 elements,
 * or b*G > 65535), ALIGN, HIP. */
int basp_pack(const void *const *src_shards, void *dst, int b, int S,
              int n_heads, int d, int G, int rank, basp_dtype dtype, void *stream);

/* Send side, the inverse on the rank's head slice (Sec. II-C: the second
 * all-to-all returns the attention output to the sequence owners):
 *   dst_shards[j][beta][t][rank*n/G + h][e] = src[beta][j*S/G + t][h][e]
 * Heads outside [rank*n/G, (rank+1)*n/G) of every dst shard are left
 * untouched.  Arguments and errors as basp_pack, plus SHAPE when n < G (a
 * shared head takes basp_unpack_add). */
int basp_unpack(const void *src, void *const *dst_shards, int b, int S,
                int n_heads, int d, int G, int rank, basp_dtype dtype, void *stream);

/* Gradient form of basp_unpack, fp32 only: the rank's rows are added into
 * the shards instead of written,
 *   dst_shards[j][beta][t][rank*n/G + h][e] += src[beta][j*S/G + t][h][e]
 * so that the G/n members sharing a kv head (n < G, Sec. II-A GQA under the
 * head split of Sec. II-C) accumulate dK and dV of that head; with n a
 * multiple of G it adds the rank's disjoint slice.  The caller clears the
 * shards first; calls for members that share a head must not overlap on
 * the device (each reads and writes the same rows; issue them in member
 * order on one stream for a deterministic sum).  src: device [b, S, nl, d]
 * fp32; shards as basp_pack with 4-byte elements.  Errors as basp_pack. */
int basp_unpack_add(const float *src, float *const *dst_shards, int b, int S,
                    int n_heads, int d, int G, int rank, void *stream);

/* The receive side of a step's first exchange in one call (Sec. II-C: Q, K
 * and V are exchanged together): the same as basp_pack of Q (n = H), then
 * of K and V (n = H_kv), bit for bit, with one kernel launch for all three
 * when G <= 16 and the rows allow the same access width (small K and V packs
 * then do not each pay a launch).  q, k, v: device [b, S, H/G, d] and
 * [b, S, Hkl, d] (Hkl as for basp_attn_fwd).  Errors: those of the three
 * basp_pack calls, checked before anything is launched. */
int basp_pack_qkv(const void *const *q_shards, const void *const *k_shards,
                  const void *const *v_shards, void *q, void *k, void *v, int b,
                  int S, int H, int H_kv, int d, int G, int rank, basp_dtype dtype,
                  void *stream);

/* The send side of the backward's last exchange in one call: basp_unpack of
 * dQ (n = H), then of dK and dV (n = H_kv), fp32, bit for bit, as one launch
 * under the conditions of basp_pack_qkv.  When H_kv < G the rank's kv head is
 * shared and dK, dV are added into the shards as basp_unpack_add does (the
 * caller clears them first).  Errors: those of the three unpacks. */
int basp_unpack_grads(const float *dq, const float *dk, const float *dv,
                      float *const *dq_shards, float *const *dk_shards,
                      float *const *dv_shards, int b, int S, int H, int H_kv,
                      int d, int G, int rank, void *stream);

/* Send side of the first all-to-all, on the owner of a sequence shard
 * (Sec. II-C: every member sends each other member that member's share of
 * the heads; Sec. IV-C runs it inside a batch-aware group): the own shard,
 * all heads, split into one contiguous block per destination member j,
 *   send[j][beta][t][h][e] = own[beta][t][j*n/G + h][e]
 * own: device [b, S/G, n, d]; send: device [G, b, S/G, n/G, d], so block j is
 * one contiguous run of b*(S/G)*(n/G)*d elements for the exchange.  With the
 * blocks of every member received, the head-sharded tensor basp_pack builds
 * is block j at rows j*S/G .. of each sequence (for b = 1, the received
 * buffer itself).  With n < G, block j holds the one head j*n/G
 * (send [G, b, S/G, 1, d]).  dtype as basp_pack; values copied bit for bit.
 * Errors: NULL, SHAPE (as basp_pack), UNSUPPORTED (as basp_pack), ALIGN, HIP. */
int basp_a2a_pack(const void *own, void *send, int b, int S, int n_heads, int d,
                  int G, basp_dtype dtype, void *stream);

/* Receive side of the second all-to-all (the attention output returns to
 * the sequence owners): block j, received from member j and holding heads
 * [j*n/G, (j+1)*n/G) of the own tokens, into the own shard:
 *   own[beta][t][j*n/G + h][e] = recv[j][beta][t][h][e]
 * recv: device [G, b, S/G, n/G, d]; own: device [b, S/G, n, d].  With n < G
 * (gradients of shared kv heads, fp32 only) recv is [G, b, S/G, 1, d] and
 * each head is the sum of its members' blocks, taken in member order:
 *   own[beta][t][h][e] = recv[h*G/n][..] + recv[h*G/n + 1][..] + ...
 * Arguments and errors as basp_a2a_pack, plus UNSUPPORTED for a bf16 tensor
 * with n < G. */
int basp_a2a_unpack(const void *recv, void *own, int b, int S, int n_heads, int d,
                    int G, basp_dtype dtype, void *stream);

/* basp_a2a_pack of an fp32 tensor with the conversion to bf16 fused, so that
 * a gradient kept in fp32 crosses the exchange at half the bytes (Sec. II-C:
 * in the backward the sequence owner sends its dO shard through the same
 * all-to-all as Q in the forward; mixed-precision training, Sec. V):
 *   send[j][beta][t][h][e] = bf16(own[beta][t][j*n/G + h][e])
 * bf16() rounds to nearest even (infinities stay infinite; NaN stays NaN).
 * own: device [b, S/G, n, d] fp32, 4-byte aligned; send: device
 * [G, b, S/G, n/G, d] bf16 (with n < G: [G, b, S/G, 1, d], block j holding
 * head j*n/G), 2-byte aligned.  16/8-byte aligned pointers and row lengths
 * that are multiples of 4 elements move 4 elements at a time.
 * Errors: NULL, SHAPE and UNSUPPORTED as basp_a2a_pack, ALIGN, HIP. */
int basp_a2a_pack_bf16(const float *own, void *send, int b, int S, int n_heads,
                       int d, int G, void *stream);

/* Causal GQA scaled dot-product attention (Sec. II-A) over the full sequence
 * for the rank's H/G query heads:
 *   O_i = sum_{j<=i} softmax_j(scale * q_i . k_j) v_j,
 *   LSE_i = log sum_{j<=i} exp(scale * q_i . k_j).
 * q [b,S,H/G,d], k/v [b,S,Hkl,d] bf16 in (Hkl = H_kv/G, or 1 when H_kv < G
 * divides G); o [b,S,H/G,d] bf16 out,
 * lse [b,H/G,S] fp32 out (kept for the backward).  bf16 MFMA products with
 * fp32 accumulation and an fp32 online softmax.
 * Alignment: q, k, v, o 16 bytes; lse 4 bytes.
 * Head dims 64, 80, 96 and 128 (the Table II models' hidden size / heads);
 * 80 is computed at width 96 with zero padding, which changes nothing in the
 * result.
 * Errors: NULL, SHAPE, UNSUPPORTED (d not 64, 80, 96 or 128, scale not
 * finite and positive, S*(H/G)*d*2 >= 2^31 bytes, b*S >= 2^31 - 1, or
 * b > 65535), ALIGN, HIP. */
int basp_attn_fwd(const void *q, const void *k, const void *v, void *o,
                  float *lse, int b, int S, int H, int H_kv, int d, int G,
                  float scale, void *stream);

/* basp_attn_fwd on the exchange's buffers in place (Sec. II-C with
 * Sec. II-A): Q, K, V are read from the G sequence shards the first
 * all-to-all delivers and O is written into the rank's head slice of the G
 * shard buffers of the second, with no pack or unpack pass:
 *   o_shards[j][beta][t][rank*H/G + h][e] = O[beta][j*S/G + t][h][e]
 * for O the attention of the rank's heads over the whole sequence.  The
 * result is bit for bit that of basp_pack, basp_attn_fwd, basp_unpack.
 * q_shards, o_shards: host arrays of G device pointers, each [b, S/G, H, d]
 * bf16; k_shards, v_shards: each [b, S/G, H_kv, d] bf16 (the rank reads kv
 * heads [rank*H_kv/G, ..), or the one shared head when H_kv < G); lse
 * [b, H/G, S] fp32 as basp_attn_fwd.  Heads of o_shards outside the rank's
 * slice are untouched.  Alignment: every shard pointer 16 bytes, lse 4.
 * Errors: as basp_attn_fwd, plus RANK, and UNSUPPORTED when G > 64, S/G is
 * not a multiple of 256, or (S/G)*max(H, H_kv)*d*4 >= 2^31 bytes. */
int basp_attn_fwd_sharded(const void *const *q_shards,
                          const void *const *k_shards,
                          const void *const *v_shards, void *const *o_shards,
                          float *lse, int b, int S, int H, int H_kv, int d,
                          int G, int rank, float scale, void *stream);

/* Bytes of device workspace basp_attn_bwd (and basp_attn_bwd_sharded) needs
 * for this share of the Sec. II-A attention backward: the per-row pair
 * (LSE, D_i = dO_i . O_i) of every local query head, and, when S is longer
 * than one row chunk of the key pass (a quarter of S, 2048 to 8192 rows;
 * past S = 128K a sixteenth of S, so never more than 16 chunks and a
 * workspace linear in S), fp32 partial sums of dK and dV per chunk.  0 for
 * an invalid shape, and
 * for an empty one (b == 0 or S == 0), which needs none. */
size_t basp_attn_bwd_workspace_bytes(int b, int S, int H, int H_kv, int d,
                                     int G);

/* Backward of basp_attn_fwd (the Sec. II-A scaled dot-product attention;
 * the paper states the forward, and the gradients follow from it):
 *   P_ij = exp(scale q_i.k_j - LSE_i),  D_i = dO_i . O_i,
 *   dS_ij = P_ij (dO_i . v_j - D_i),
 *   dQ_i = scale sum_{j<=i} dS_ij k_j,
 *   dK_j = scale sum_{h} sum_{i>=j} dS_ij q_i,  dV_j = sum_{h} sum_{i>=j} P_ij dO_i
 * (h over the local query heads of kv head j's group), for the loss
 * sum(O * dO): inputs q, k, v, o, d_o
 * (bf16, layouts as above) and lse from the forward; outputs
 * dq [b,S,H/G,d], dk/dv [b,S,Hkl,d] in fp32, each fully overwritten
 * (dk/dv sum over the rank's query heads sharing a kv head; with a kv head
 * shared by several members these are that member's part).  workspace:
 * device buffer of at least basp_attn_bwd_workspace_bytes(), 16-byte
 * aligned, contents ignored on entry and undefined on return.  Results are
 * deterministic (no atomics).
 * Errors: NULL, SHAPE, UNSUPPORTED, ALIGN, WORKSPACE, HIP. */
int basp_attn_bwd(const void *q, const void *k, const void *v, const void *o,
                  const float *lse, const void *d_o, float *dq, float *dk,
                  float *dv, void *workspace, size_t workspace_bytes, int b,
                  int S, int H, int H_kv, int d, int G, float scale,
                  void *stream);

/* Size of the device scratch buffer basp_attn_bwd_noalloc uses instead of a
 * workspace argument (128 MiB, held on each GPU the library runs on). */
#define BASP_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)

/* basp_attn_bwd for callers that cannot allocate device memory (code under
 * stream capture, allocation-free serving loops, harnesses that forbid
 * hipMalloc): the same computation and results, bit for bit, with the
 * workspace taken from a static device buffer of BASP_NOALLOC_SCRATCH_BYTES
 * that the library holds on each GPU.  The first call on a GPU looks up that
 * buffer's address; no call allocates or frees anything.  Arguments as
 * basp_attn_bwd without workspace/workspace_bytes; the device is the one
 * `stream` belongs to (the current device for the null stream).  Calls on
 * one GPU share its buffer: calls that overlap on the device (other streams,
 * other host threads) race and must not be issued; calls in order on one
 * stream are safe, since nothing in the buffer is carried from one call to
 * the next.  Errors: as basp_attn_bwd, and BASP_ERR_WORKSPACE when the shape
 * needs more than BASP_NOALLOC_SCRATCH_BYTES
 * (basp_attn_bwd_workspace_bytes() tells how much it needs), HIP when the
 * buffer's address cannot be obtained. */
int basp_attn_bwd_noalloc(const void *q, const void *k, const void *v,
                          const void *o, const float *lse, const void *d_o,
                          float *dq, float *dk, float *dv, int b, int S, int H,
                          int H_kv, int d, int G, float scale, void *stream);

/* basp_attn_bwd on the exchange's buffers in place: Q, K, V, O and dO are
 * read from their G sequence shards (layouts as basp_attn_fwd_sharded; dO as
 * Q) and dQ, dK, dV (fp32) are written into the rank's head slices of their
 * G shard buffers ([b, S/G, H, d] for dQ, [b, S/G, H_kv, d] for dK and dV);
 * other heads are untouched.  The result is bit for bit that of basp_pack
 * (of dO), basp_attn_bwd and basp_unpack of each gradient.  lse as there;
 * workspace of basp_attn_bwd_sharded_workspace_bytes(), 16-byte aligned
 * (the rank's heads of Q, dO, K and V are first packed into it: the passes
 * stream those rows many times, and local rows stream faster than rows a
 * whole shard row apart).
 * With a kv head shared by G/H_kv members (H_kv < G, Sec. II-A GQA under the
 * head split of Sec. II-C) each member holds only a partial dK, dV of that
 * head, which the reverse exchange must sum: dk_shards and dv_shards are
 * then G send blocks, block j [b, S/G, 1, d] receiving this member's partial
 * gradient of member j's tokens (bit for bit rows j*S/G .. of basp_attn_bwd's
 * dk, dv); member j sums the blocks of the sharing members in member order
 * (basp_a2a_unpack does this).
 * Errors: as basp_attn_fwd_sharded, plus WORKSPACE. */
/* Bytes of device workspace basp_attn_bwd_sharded needs: local copies of
 * the rank's heads of Q and dO (each [b, S, H/G, d] bf16) and of K and V
 * (each [b, S, Hkl, d] bf16, Hkl as basp_attn_fwd), each rounded up to 256
 * bytes, then basp_attn_bwd_workspace_bytes().  0 for an invalid or empty
 * shape. */
size_t basp_attn_bwd_sharded_workspace_bytes(int b, int S, int H, int H_kv,
                                             int d, int G);

int basp_attn_bwd_sharded(const void *const *q_shards,
                          const void *const *k_shards,
                          const void *const *v_shards,
                          const void *const *o_shards, const float *lse,
                          const void *const *do_shards, float *const *dq_shards,
                          float *const *dk_shards, float *const *dv_shards,
                          void *workspace, size_t workspace_bytes, int b,
                          int S, int H, int H_kv, int d, int G, int rank,
                          float scale, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* BASP_H */
