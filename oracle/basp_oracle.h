/*
 * basp_oracle.h -- plain CPU reference for one rank's share of batch-aware
 * Ulysses attention (BASP, "Batch-Aware Sequence Parallelism for LLM
 * Training", Sec. II-A, Sec. II-C, Sec. IV, Alg. 1, Alg. 2).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header or helper with the HIP library; the product path never calls it.
 *
 * Everything is fp64 (attention) or raw bytes (permutations), slow and plain.
 * Layouts (row-major, innermost last):
 *   sequence shard       [b, S/G, n, d]    one per group member j
 *   head-sharded local   [b, S, n/G, d]
 *   LSE                  [b, Hl, rows]     natural logarithm
 * Return value of the int functions: 0 on success, a negative code on bad
 * arguments (see basp_oracle.c).
 */
#ifndef BASP_ORACLE_H
#define BASP_ORACLE_H

#ifdef __cplusplus
extern "C" {
#endif

/* Alg. 1 (group formation) and Alg. 2 (rank -> group, local rank). */
int oracle_group_of(long world, long micro_batch, long global_rank,
                    long *group, long *local_rank, long *group_size);

/* Alg. 2: which sequence and which token range a global rank holds. */
int oracle_seq_partition(long L, long K, long global_rank,
                         long *seq_start, long *seq_end,
                         long *tok_start, long *tok_end);

/* Receive side of the Ulysses all-to-all, all G sources at once (Sec. II-C):
 * dst[beta][j*S/G + t][h][e] = src_j[beta][t][rank*n/G + h][e].
 * elem = bytes per element (2 or 4); copied as raw bytes. */
int oracle_pack(const void *const *src, void *dst, long b, long S, long n,
                long d, long G, long rank, long elem);

/* Inverse on the rank's head slice; every other head of dst_j is untouched.
 * Needs G | n. */
int oracle_unpack(const void *src, void *const *dst, long b, long S, long n,
                  long d, long G, long rank, long elem);

/* Head slices: with G | n, member `rank` handles heads [rank*n/G, +n/G);
 * with n < G and n | G (fewer kv heads than members, Sec. II-A's GQA under
 * Ulysses' head split), the one head rank*n/G, shared by G/n members.
 * oracle_pack above follows this rule.  The fp32 variant of unpack that
 * adds the rank's part into the shards, for gradients of a shared head:
 *   dst_j[beta][t][h0 + h][e] += src[beta][j*S/G + t][h][e]. */
int oracle_unpack_add(const float *src, float *const *dst, long b, long S,
                      long n, long d, long G, long rank);

/* Send side of the all-to-all, on the owner of a sequence shard (Sec. II-C:
 * each member sends every other member its share of the heads): the own
 * shard [b, S/G, n, d], all heads, split by destination member j into
 *   send[j][beta][t][h][e] = own[beta][t][j*n/G + h][e],  send [G, b, S/G, n/G, d]
 * (with n < G: the one head j*n/G, send [G, b, S/G, 1, d]).
 * elem = bytes per element (2 or 4); copied as raw bytes. */
int oracle_a2a_pack(const void *own, void *send, long b, long S, long n,
                    long d, long G, long elem);

/* Receive side of the reverse all-to-all (the output goes back to the
 * sequence owners): block j, the heads [j*n/G, (j+1)*n/G) member j computed,
 * into the own shard:
 *   own[beta][t][j*n/G + h][e] = recv[j][beta][t][h][e],  recv [G, b, S/G, n/G, d].
 * With n < G (fp32 only): head h is the sum, in member order, of the blocks
 * of the G/n members that share it. */
int oracle_a2a_unpack(const void *recv, void *own, long b, long S, long n,
                      long d, long G, long elem);

/* oracle_a2a_pack of an fp32 own shard with every element converted to bf16
 * by round to nearest even (raw bf16 bit patterns out). */
int oracle_a2a_pack_bf16(const float *own, unsigned short *send, long b, long S,
                         long n, long d, long G);

/* Causal scaled dot-product attention (Sec. II-A), local q head h reads local
 * kv head h / (Hl/Hkl).  Computes rows [r0, r1) of every (beta, h):
 *   o   [b, r1-r0, Hl, d],  lse [b, Hl, r1-r0].
 * q [b,S,Hl,d], k/v [b,S,Hkl,d] are full tensors. */
int oracle_attn_fwd(const double *q, const double *k, const double *v,
                    double *o, double *lse, long b, long S, long Hl, long Hkl,
                    long d, double scale, long r0, long r1);

/* Backward of the above for the loss sum(O * dO).  o/lse are rows [r0, S)
 * from oracle_attn_fwd(r0, S).  Produces exact gradients for query rows and
 * key rows in [r0, S):  dq [b,S-r0,Hl,d], dk/dv [b,S-r0,Hkl,d]. */
int oracle_attn_bwd(const double *q, const double *k, const double *v,
                    const double *dout, const double *o, const double *lse,
                    double *dq, double *dk, double *dv, long b, long S,
                    long Hl, long Hkl, long d, double scale, long r0);

/* Row-local results for a list of (beta, head, row) samples: O_i, LSE_i and
 * dQ_i, each needing only keys j <= i.  o_out/dq_out [n, d], lse_out [n]. */
int oracle_attn_rows(const double *q, const double *k, const double *v,
                     const double *dout, long b, long S, long Hl, long Hkl,
                     long d, double scale, long nsamp, const long *beta,
                     const long *head, const long *row, double *o_out,
                     double *lse_out, double *dq_out);

/* Key-local results for a list of (beta, kv head, key) samples: dK_j and
 * dV_j summed over the query heads of the kv head and over every row i >= j.
 * o [b,S,Hl,d] and lse [b,Hl,S] are all rows of oracle_attn_fwd.
 * dk_out/dv_out [n, d]. */
int oracle_attn_keys(const double *q, const double *k, const double *v,
                     const double *dout, const double *o, const double *lse,
                     long b, long S, long Hl, long Hkl, long d, double scale,
                     long nsamp, const long *beta, const long *kvhead,
                     const long *key, double *dk_out, double *dv_out);

/* Number of OpenMP threads the oracle runs with. */
int oracle_threads(void);

/* Set the number of OpenMP threads (n < 1: all available processors). */
void oracle_set_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
