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
 *   basp_a2a_pack / basp_a2a_unpack   the owner's side of the same exchanges:
 *                  own shard <-> one contiguous block per member
 *
 * The exchange itself (RCCL) is not part of this library.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Shapes (row-major, innermost last; "n" is the global head count of the
 * tensor at hand: H for Q, O, dO, dQ and H_kv for K, V, dK, dV):
 *   sequence shard j      [b, S/G, n,   d]   tokens [j*S/G, (j+1)*S/G)
 *   head-sharded local    [b, S,   n/G, d]   heads  [rank*n/G, (rank+1)*n/G)
 *   LSE                   [b, H/G, S]        fp32, natural logarithm
 * GQA: local query head h attends with local kv head h / (H/H_kv); the
 * rank's kv heads are the contiguous block [rank*H_kv/G, (rank+1)*H_kv/G).
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
  BASP_ERR_SHAPE = 2,       /* negative size, or S%G, H%G, H_kv%G, H%H_kv != 0 */
  BASP_ERR_RANK = 3,        /* rank outside [0, G)                           */
  BASP_ERR_UNSUPPORTED = 4, /* d, dtype, G or size outside what the kernels handle */
  BASP_ERR_ALIGN = 5,       /* pointer not aligned as documented             */
  BASP_ERR_WORKSPACE = 6,   /* workspace smaller than the query reports      */
  BASP_ERR_HIP = 7,         /* a HIP launch failed                           */
  BASP_ERR_DP_FALLBACK = 8  /* micro-batch larger than the world (plain DP)  */
} basp_status;

typedef enum basp_dtype { BASP_BF16 = 0, BASP_F32 = 1 } basp_dtype;

/* Largest group size the permutation kernels accept. */
#define BASP_MAX_GROUP 128

/* Human-readable name of a status code (static string, never NULL). */
const char *basp_status_str(int status);

/* Batch-aware group formation (Alg. 1) and rank placement (Alg. 2):
 * world N GPUs, micro-batch B; K = N/B, groups of K contiguous ranks,
 * group = floor(rank/K), local_rank = rank mod K.  Host only.
 * Errors: SHAPE (N or B < 1, N % B != 0), DP_FALLBACK (B > N),
 * RANK (global_rank outside [0, N)), NULL. */
int basp_group_of(int world, int micro_batch, int global_rank, int *group,
                  int *local_rank, int *group_size);

/* Check a share's parameters (b, S, H, H_kv, d, G, rank) without touching
 * the GPU.  Returns BASP_OK or the code the other entry points would give
 * for the same shape (UNSUPPORTED when d is not 64, 80, 96 or 128). */
int basp_validate(int b, int S, int H, int H_kv, int d, int G, int rank);

/* Receive side of the head-parallel all-to-all (Sec. II-C, Sec. IV-C):
 *   dst[beta][j*S/G + t][h][e] = src_shards[j][beta][t][rank*n/G + h][e]
 * src_shards: host array of G device pointers, each [b, S/G, n, d];
 * dst: device [b, S, n/G, d].  dtype selects 2-byte (BASP_BF16) or 4-byte
 * (BASP_F32) elements; values are copied bit for bit.
 * Alignment: every pointer aligned to the element size.
 * Errors: NULL, SHAPE, RANK, UNSUPPORTED (dtype, G > BASP_MAX_GROUP,
 * (S/G)*(n/G)*d >= 2^31 elements, or b*G > 65535), ALIGN, HIP. */
int basp_pack(const void *const *src_shards, void *dst, int b, int S,
              int n_heads, int d, int G, int rank, int dtype, void *stream);

/* Send side, the inverse on the rank's head slice (Sec. II-C: the second
 * all-to-all returns the attention output to the sequence owners):
 *   dst_shards[j][beta][t][rank*n/G + h][e] = src[beta][j*S/G + t][h][e]
 * Heads outside [rank*n/G, (rank+1)*n/G) of every dst shard are left
 * untouched.  Arguments and errors as basp_pack. */
int basp_unpack(const void *src, void *const *dst_shards, int b, int S,
                int n_heads, int d, int G, int rank, int dtype, void *stream);

/* Send side of the first all-to-all, on the owner of a sequence shard
 * (Sec. II-C: every member sends each other member that member's share of
 * the heads; Sec. IV-C runs it inside a batch-aware group): the own shard,
 * all heads, split into one contiguous block per destination member j,
 *   send[j][beta][t][h][e] = own[beta][t][j*n/G + h][e]
 * own: device [b, S/G, n, d]; send: device [G, b, S/G, n/G, d], so block j is
 * one contiguous run of b*(S/G)*(n/G)*d elements for the exchange.  With the
 * blocks of every member received, the head-sharded tensor basp_pack builds
 * is block j at rows j*S/G .. of each sequence (for b = 1, the received
 * buffer itself).  dtype as basp_pack; values copied bit for bit.
 * Errors: NULL, SHAPE (S % G, n % G), UNSUPPORTED (as basp_pack), ALIGN, HIP. */
int basp_a2a_pack(const void *own, void *send, int b, int S, int n_heads, int d,
                  int G, int dtype, void *stream);

/* Receive side of the second all-to-all (the attention output returns to
 * the sequence owners): block j, received from member j and holding heads
 * [j*n/G, (j+1)*n/G) of the own tokens, into the own shard:
 *   own[beta][t][j*n/G + h][e] = recv[j][beta][t][h][e]
 * recv: device [G, b, S/G, n/G, d]; own: device [b, S/G, n, d].  Arguments
 * and errors as basp_a2a_pack. */
int basp_a2a_unpack(const void *recv, void *own, int b, int S, int n_heads, int d,
                    int G, int dtype, void *stream);

/* Causal GQA scaled dot-product attention (Sec. II-A) over the full sequence
 * for the rank's H/G query heads:
 *   O_i = sum_{j<=i} softmax_j(scale * q_i . k_j) v_j,
 *   LSE_i = log sum_{j<=i} exp(scale * q_i . k_j).
 * q [b,S,H/G,d], k/v [b,S,H_kv/G,d] bf16 in; o [b,S,H/G,d] bf16 out,
 * lse [b,H/G,S] fp32 out (kept for the backward).  bf16 MFMA products with
 * fp32 accumulation and an fp32 online softmax.
 * Alignment: q, k, v, o 16 bytes; lse 4 bytes.
 * Head dims 64, 80, 96 and 128 (the Table II models' hidden size / heads);
 * 80 is computed at width 96 with zero padding, which changes nothing in the
 * result.
 * Errors: NULL, SHAPE, UNSUPPORTED (d not 64, 80, 96 or 128, scale not
 * finite and positive, or S*(H/G)*d*2 >= 2^31 bytes), ALIGN, HIP. */
int basp_attn_fwd(const void *q, const void *k, const void *v, void *o,
                  float *lse, int b, int S, int H, int H_kv, int d, int G,
                  float scale, void *stream);

/* Bytes of device workspace basp_attn_bwd needs for this shape. */
size_t basp_attn_bwd_workspace_bytes(int b, int S, int H, int H_kv, int d,
                                     int G);

/* Backward of basp_attn_fwd for the loss sum(O * dO): inputs q, k, v, o, d_o
 * (bf16, layouts as above) and lse from the forward; outputs
 * dq [b,S,H/G,d], dk/dv [b,S,H_kv/G,d] in fp32, each fully overwritten
 * (dk/dv sum over the H/H_kv query heads sharing a kv head).  workspace:
 * device buffer of at least basp_attn_bwd_workspace_bytes(), 16-byte
 * aligned, contents ignored on entry and undefined on return.  Results are
 * deterministic (no atomics).
 * Errors: NULL, SHAPE, UNSUPPORTED, ALIGN, WORKSPACE, HIP. */
int basp_attn_bwd(const void *q, const void *k, const void *v, const void *o,
                  const float *lse, const void *d_o, float *dq, float *dk,
                  float *dv, void *workspace, size_t workspace_bytes, int b,
                  int S, int H, int H_kv, int d, int G, float scale,
                  void *stream);

#ifdef __cplusplus
}
#endif
#endif /* BASP_H */
