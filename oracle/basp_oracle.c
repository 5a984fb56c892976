/*
 * basp_oracle.c -- plain CPU reference for one rank's share of batch-aware
 * Ulysses attention.  TEST INFRASTRUCTURE ONLY (see basp_oracle.h).
 *
 * Sources in the paper:
 *   group formation ........ Alg. 1, Sec. IV-A (K = N/B, contiguous ranks)
 *   rank -> (group, local) . Alg. 2, Sec. IV-B (g = floor(r/K), l = r mod K,
 *                            contiguous token chunks of length L/K)
 *   head-parallel exchange . Sec. II-C (the all-to-all hands each rank the
 *                            full sequence for a subset of heads) and
 *                            Sec. IV-C (the same exchange inside a group)
 *   attention .............. Sec. II-A, the scaled dot-product equation,
 *                            causal mask j <= i, softmax scale given by caller
 * The backward is derived by hand from the forward definition:
 *   D_i   = sum_e dO_i[e] O_i[e]
 *   dP_ij = dO_i . v_j,   dS_ij = P_ij (dP_ij - D_i)
 *   dV_j  = sum_{h in group} sum_{i>=j} P_ij dO_i
 *   dQ_i  = c sum_{j<=i} dS_ij k_j
 *   dK_j  = c sum_{h in group} sum_{i>=j} dS_ij q_i
 * No tiling, no online softmax: two passes over each full score row.
 */
#include "basp_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum {
  ORC_OK = 0,
  ORC_ERR_SHAPE = -1,     /* a size is negative or a divisibility fails */
  ORC_ERR_RANK = -2,      /* rank outside its range */
  ORC_ERR_DP = -3,        /* micro-batch larger than world: plain data parallel */
  ORC_ERR_NULL = -4,
  ORC_ERR_ELEM = -5,
  ORC_ERR_RANGE = -6,
};

int oracle_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads of the parallel loops from now on (n < 1: every available one). */
void oracle_set_threads(int n) {
#ifdef _OPENMP
  omp_set_num_threads(n >= 1 ? n : omp_get_num_procs());
#else
  (void)n;
#endif
}

/* ---------------------------------------------------------------- Alg. 1 */
int oracle_group_of(long world, long micro_batch, long global_rank,
                    long *group, long *local_rank, long *group_size) {
  if (world < 1 || micro_batch < 1) return ORC_ERR_SHAPE;
  if (micro_batch > world) return ORC_ERR_DP;       /* Sec. IV-A fallback */
  if (world % micro_batch != 0) return ORC_ERR_SHAPE; /* the assert of Alg. 1 */
  if (global_rank < 0 || global_rank >= world) return ORC_ERR_RANK;
  long K = world / micro_batch;  /* group size */
  long num_groups = micro_batch;
  /* Walk the groups in order; group i holds ranks iK .. iK+K-1. */
  for (long i = 0; i < num_groups; ++i) {
    long first = i * K, last = i * K + K - 1;
    if (global_rank >= first && global_rank <= last) {
      *group = i;
      *local_rank = global_rank - first;
      *group_size = K;
      return ORC_OK;
    }
  }
  return ORC_ERR_RANK;
}

/* ---------------------------------------------------------------- Alg. 2 */
int oracle_seq_partition(long L, long K, long global_rank, long *seq_start,
                         long *seq_end, long *tok_start, long *tok_end) {
  if (L < 0 || K < 1 || global_rank < 0) return ORC_ERR_SHAPE;
  if (L % K != 0) return ORC_ERR_SHAPE;
  long my_group = global_rank / K;
  long my_local = global_rank % K;
  long chunk = L / K;
  *seq_start = my_group;
  *seq_end = my_group + 1;
  *tok_start = my_local * chunk;
  *tok_end = (my_local + 1) * chunk;
  return ORC_OK;
}

/* ------------------------------------------------------- pack / unpack */
/* Heads of a tensor with n heads that group member j handles: n/G of them
 * from j*n/G when G divides n; when n < G and n divides G (fewer kv heads
 * than members), the single head j*n/G (integer division), shared by the
 * G/n members j with the same quotient. */
static long first_head(long n, long G, long j) { return j * n / G; }
static long heads_per_member(long n, long G) { return n >= G ? n / G : 1; }

static int perm_args_ok(long b, long S, long n, long d, long G, long rank,
                        long elem) {
  if (b < 0 || S < 0 || n < 1 || d < 1 || G < 1) return ORC_ERR_SHAPE;
  if (S % G != 0) return ORC_ERR_SHAPE;
  if (!(n % G == 0 || (n < G && G % n == 0))) return ORC_ERR_SHAPE;
  if (rank < 0 || rank >= G) return ORC_ERR_RANK;
  if (elem != 2 && elem != 4) return ORC_ERR_ELEM;
  return ORC_OK;
}

int oracle_pack(const void *const *src, void *dst, long b, long S, long n,
                long d, long G, long rank, long elem) {
  int rc = perm_args_ok(b, S, n, d, G, rank, elem);
  if (rc) return rc;
  if (!src || !dst) return ORC_ERR_NULL;
  for (long j = 0; j < G; ++j)
    if (!src[j]) return ORC_ERR_NULL;
  long Sg = S / G, nl = heads_per_member(n, G), h0 = first_head(n, G, rank);
  for (long j = 0; j < G; ++j) {
    const unsigned char *s = (const unsigned char *)src[j];
#pragma omp parallel for collapse(2)
    for (long beta = 0; beta < b; ++beta)
      for (long t = 0; t < Sg; ++t)
        for (long h = 0; h < nl; ++h)
          for (long e = 0; e < d; ++e) {
            long from = ((beta * Sg + t) * n + (h0 + h)) * d + e;
            long to = ((beta * S + (j * Sg + t)) * nl + h) * d + e;
            memcpy((unsigned char *)dst + to * elem, s + from * elem,
                   (size_t)elem);
          }
  }
  return ORC_OK;
}

int oracle_unpack(const void *src, void *const *dst, long b, long S, long n,
                  long d, long G, long rank, long elem) {
  int rc = perm_args_ok(b, S, n, d, G, rank, elem);
  if (rc) return rc;
  if (!src || !dst) return ORC_ERR_NULL;
  if (n < G) return ORC_ERR_SHAPE; /* a shared head takes oracle_unpack_add */
  for (long j = 0; j < G; ++j)
    if (!dst[j]) return ORC_ERR_NULL;
  long Sg = S / G, nl = n / G;
  for (long j = 0; j < G; ++j) {
    unsigned char *o = (unsigned char *)dst[j];
#pragma omp parallel for collapse(2)
    for (long beta = 0; beta < b; ++beta)
      for (long t = 0; t < Sg; ++t)
        for (long h = 0; h < nl; ++h)
          for (long e = 0; e < d; ++e) {
            long from = ((beta * S + (j * Sg + t)) * nl + h) * d + e;
            long to = ((beta * Sg + t) * n + (rank * nl + h)) * d + e;
            memcpy(o + to * elem, (const unsigned char *)src + from * elem,
                   (size_t)elem);
          }
  }
  return ORC_OK;
}

int oracle_unpack_add(const float *src, float *const *dst, long b, long S, long n,
                      long d, long G, long rank) {
  int rc = perm_args_ok(b, S, n, d, G, rank, 4);
  if (rc) return rc;
  if (!src || !dst) return ORC_ERR_NULL;
  for (long j = 0; j < G; ++j)
    if (!dst[j]) return ORC_ERR_NULL;
  long Sg = S / G, nl = heads_per_member(n, G), h0 = first_head(n, G, rank);
  for (long j = 0; j < G; ++j) {
    float *o = dst[j];
#pragma omp parallel for collapse(2)
    for (long beta = 0; beta < b; ++beta)
      for (long t = 0; t < Sg; ++t)
        for (long h = 0; h < nl; ++h)
          for (long e = 0; e < d; ++e) {
            long from = ((beta * S + (j * Sg + t)) * nl + h) * d + e;
            long to = ((beta * Sg + t) * n + (h0 + h)) * d + e;
            o[to] = o[to] + src[from];
          }
  }
  return ORC_OK;
}

int oracle_a2a_pack(const void *own, void *send, long b, long S, long n,
                    long d, long G, long elem) {
  int rc = perm_args_ok(b, S, n, d, G, 0, elem);
  if (rc) return rc;
  if (!own || !send) return ORC_ERR_NULL;
  long Sg = S / G, nl = heads_per_member(n, G);
  for (long j = 0; j < G; ++j)
    for (long beta = 0; beta < b; ++beta)
      for (long t = 0; t < Sg; ++t)
        for (long h = 0; h < nl; ++h)
          for (long e = 0; e < d; ++e) {
            long from = ((beta * Sg + t) * n + (first_head(n, G, j) + h)) * d + e;
            long to = (((j * b + beta) * Sg + t) * nl + h) * d + e;
            memcpy((unsigned char *)send + to * elem,
                   (const unsigned char *)own + from * elem, (size_t)elem);
          }
  return ORC_OK;
}

int oracle_a2a_unpack(const void *recv, void *own, long b, long S, long n,
                      long d, long G, long elem) {
  int rc = perm_args_ok(b, S, n, d, G, 0, elem);
  if (rc) return rc;
  if (!recv || !own) return ORC_ERR_NULL;
  long Sg = S / G;
  if (n < G) {
    /* Shared heads: head h is the sum of the blocks of its G/n members, in
     * member order (fp32 partial gradients). */
    if (elem != 4) return ORC_ERR_ELEM;
    const float *r = (const float *)recv;
    float *o = (float *)own;
    for (long h = 0; h < n; ++h)
      for (long beta = 0; beta < b; ++beta)
        for (long t = 0; t < Sg; ++t)
          for (long e = 0; e < d; ++e) {
            float acc = 0.0f;
            int first = 1;
            for (long j = 0; j < G; ++j) {
              if (first_head(n, G, j) != h) continue;
              float x = r[((j * b + beta) * Sg + t) * d + e];
              acc = first ? x : acc + x;
              first = 0;
            }
            o[((beta * Sg + t) * n + h) * d + e] = acc;
          }
    return ORC_OK;
  }
  long nl = n / G;
  for (long j = 0; j < G; ++j)
    for (long beta = 0; beta < b; ++beta)
      for (long t = 0; t < Sg; ++t)
        for (long h = 0; h < nl; ++h)
          for (long e = 0; e < d; ++e) {
            long from = (((j * b + beta) * Sg + t) * nl + h) * d + e;
            long to = ((beta * Sg + t) * n + (j * nl + h)) * d + e;
            memcpy((unsigned char *)own + to * elem,
                   (const unsigned char *)recv + from * elem, (size_t)elem);
          }
  return ORC_OK;
}

/* fp32 -> bf16, round to nearest even: keep the upper 16 bits after adding
 * half an ulp of the result, minus one when the kept part is even (so that a
 * tie rounds to the even neighbour).  Infinities stay infinite and finite
 * values too large for bf16 become infinite, as rounding defines; a NaN
 * becomes the quiet NaN with the same sign. */
static unsigned short bf16_rne(float x) {
  unsigned int u;
  memcpy(&u, &x, sizeof u);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu) != 0)
    return (unsigned short)((u >> 16) | 0x0040u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (unsigned short)(u >> 16);
}

int oracle_a2a_pack_bf16(const float *own, unsigned short *send, long b, long S,
                         long n, long d, long G) {
  int rc = perm_args_ok(b, S, n, d, G, 0, 4);
  if (rc) return rc;
  if (!own || !send) return ORC_ERR_NULL;
  long Sg = S / G, nl = heads_per_member(n, G);
  for (long j = 0; j < G; ++j)
    for (long beta = 0; beta < b; ++beta)
      for (long t = 0; t < Sg; ++t)
        for (long h = 0; h < nl; ++h)
          for (long e = 0; e < d; ++e) {
            long from = ((beta * Sg + t) * n + (first_head(n, G, j) + h)) * d + e;
            long to = (((j * b + beta) * Sg + t) * nl + h) * d + e;
            send[to] = bf16_rne(own[from]);
          }
  return ORC_OK;
}

/* ------------------------------------------------------------ attention */
static double dot(const double *x, const double *y, long d) {
  double acc = 0.0;
#pragma omp simd reduction(+ : acc)
  for (long e = 0; e < d; ++e) acc += x[e] * y[e];
  return acc;
}

static int attn_args_ok(long b, long S, long Hl, long Hkl, long d) {
  if (b < 0 || S < 0 || Hl < 1 || Hkl < 1 || d < 1) return ORC_ERR_SHAPE;
  if (Hl % Hkl != 0) return ORC_ERR_SHAPE;
  return ORC_OK;
}

/* Row i of head h of sequence beta: scores s[0..i], then softmax, then P V.
 * Writes o_i[d] and returns lse_i. */
static double fwd_row(const double *q, const double *k, const double *v,
                      double *o_i, double *s, long S, long Hl, long Hkl,
                      long d, double scale, long beta, long h, long i) {
  long n_rep = Hl / Hkl, kvh = h / n_rep;
  const double *qi = q + ((beta * S + i) * Hl + h) * d;
  double m = -INFINITY;
  for (long j = 0; j <= i; ++j) {
    s[j] = scale * dot(qi, k + ((beta * S + j) * Hkl + kvh) * d, d);
    if (s[j] > m) m = s[j];
  }
  double l = 0.0;
  for (long j = 0; j <= i; ++j) {
    s[j] = exp(s[j] - m);
    l += s[j];
  }
  for (long e = 0; e < d; ++e) o_i[e] = 0.0;
  for (long j = 0; j <= i; ++j) {
    double p = s[j] / l;
    const double *vj = v + ((beta * S + j) * Hkl + kvh) * d;
    for (long e = 0; e < d; ++e) o_i[e] += p * vj[e];
  }
  return m + log(l);
}

int oracle_attn_fwd(const double *q, const double *k, const double *v,
                    double *o, double *lse, long b, long S, long Hl, long Hkl,
                    long d, double scale, long r0, long r1) {
  int rc = attn_args_ok(b, S, Hl, Hkl, d);
  if (rc) return rc;
  if (r0 < 0 || r1 > S || r0 > r1) return ORC_ERR_RANGE;
  if (!q || !k || !v || !o || !lse) return ORC_ERR_NULL;
  long R = r1 - r0;
#pragma omp parallel
  {
    double *s = (double *)malloc(sizeof(double) * (size_t)(S > 0 ? S : 1));
#pragma omp for collapse(3) schedule(dynamic, 4)
    for (long beta = 0; beta < b; ++beta)
      for (long h = 0; h < Hl; ++h)
        for (long r = 0; r < R; ++r) {
          long i = r0 + r;
          double *oi = o + ((beta * R + r) * Hl + h) * d;
          lse[(beta * Hl + h) * R + r] =
              fwd_row(q, k, v, oi, s, S, Hl, Hkl, d, scale, beta, h, i);
        }
    free(s);
  }
  return ORC_OK;
}

int oracle_attn_bwd(const double *q, const double *k, const double *v,
                    const double *dout, const double *o, const double *lse,
                    double *dq, double *dk, double *dv, long b, long S,
                    long Hl, long Hkl, long d, double scale, long r0) {
  int rc = attn_args_ok(b, S, Hl, Hkl, d);
  if (rc) return rc;
  if (r0 < 0 || r0 > S) return ORC_ERR_RANGE;
  if (!q || !k || !v || !dout || !o || !lse || !dq || !dk || !dv)
    return ORC_ERR_NULL;
  long R = S - r0, n_rep = Hl / Hkl;

  /* D_i = dO_i . O_i for the rows [r0, S). */
  double *D = (double *)malloc(sizeof(double) * (size_t)(b * Hl * R + 1));
  if (!D) return ORC_ERR_SHAPE;
#pragma omp parallel for collapse(3)
  for (long beta = 0; beta < b; ++beta)
    for (long h = 0; h < Hl; ++h)
      for (long r = 0; r < R; ++r) {
        long i = r0 + r;
        D[(beta * Hl + h) * R + r] =
            dot(dout + ((beta * S + i) * Hl + h) * d,
                o + ((beta * R + r) * Hl + h) * d, d);
      }

  /* dQ_i = c sum_{j<=i} dS_ij k_j, one query row per task. */
#pragma omp parallel for collapse(3) schedule(dynamic, 4)
  for (long beta = 0; beta < b; ++beta)
    for (long h = 0; h < Hl; ++h)
      for (long r = 0; r < R; ++r) {
        long i = r0 + r, kvh = h / n_rep;
        const double *qi = q + ((beta * S + i) * Hl + h) * d;
        const double *doi = dout + ((beta * S + i) * Hl + h) * d;
        double Li = lse[(beta * Hl + h) * R + r];
        double Di = D[(beta * Hl + h) * R + r];
        double *dqi = dq + ((beta * R + r) * Hl + h) * d;
        for (long e = 0; e < d; ++e) dqi[e] = 0.0;
        for (long j = 0; j <= i; ++j) {
          const double *kj = k + ((beta * S + j) * Hkl + kvh) * d;
          const double *vj = v + ((beta * S + j) * Hkl + kvh) * d;
          double p = exp(scale * dot(qi, kj, d) - Li);
          double ds = p * (dot(doi, vj, d) - Di);
          for (long e = 0; e < d; ++e) dqi[e] += scale * ds * kj[e];
        }
      }

  /* dK_j, dV_j: sum over the q heads sharing kv head and all rows i >= j. */
#pragma omp parallel for collapse(3) schedule(dynamic, 4)
  for (long beta = 0; beta < b; ++beta)
    for (long kvh = 0; kvh < Hkl; ++kvh)
      for (long r = 0; r < R; ++r) {
        long j = r0 + r;
        const double *kj = k + ((beta * S + j) * Hkl + kvh) * d;
        const double *vj = v + ((beta * S + j) * Hkl + kvh) * d;
        double *dkj = dk + ((beta * R + r) * Hkl + kvh) * d;
        double *dvj = dv + ((beta * R + r) * Hkl + kvh) * d;
        for (long e = 0; e < d; ++e) dkj[e] = dvj[e] = 0.0;
        for (long h = kvh * n_rep; h < (kvh + 1) * n_rep; ++h)
          for (long i = j; i < S; ++i) {
            long ri = i - r0;
            const double *qi = q + ((beta * S + i) * Hl + h) * d;
            const double *doi = dout + ((beta * S + i) * Hl + h) * d;
            double p = exp(scale * dot(qi, kj, d) - lse[(beta * Hl + h) * R + ri]);
            double ds = p * (dot(doi, vj, d) - D[(beta * Hl + h) * R + ri]);
            for (long e = 0; e < d; ++e) {
              dvj[e] += p * doi[e];
              dkj[e] += scale * ds * qi[e];
            }
          }
      }
  free(D);
  return ORC_OK;
}

/* Key-local gradients for sampled (beta, kv head, key) triples: dK_j and
 * dV_j of the definition above, summed over the query heads sharing the kv
 * head and over every row i >= j.  o/lse are all rows [0, S) of the
 * forward; D_i is formed from them row by row. */
int oracle_attn_keys(const double *q, const double *k, const double *v,
                     const double *dout, const double *o, const double *lse,
                     long b, long S, long Hl, long Hkl, long d, double scale,
                     long nsamp, const long *beta, const long *kvhead,
                     const long *key, double *dk_out, double *dv_out) {
  int rc = attn_args_ok(b, S, Hl, Hkl, d);
  if (rc) return rc;
  if (nsamp < 0) return ORC_ERR_RANGE;
  if (!q || !k || !v || !dout || !o || !lse || !beta || !kvhead || !key ||
      !dk_out || !dv_out)
    return ORC_ERR_NULL;
  for (long n = 0; n < nsamp; ++n)
    if (beta[n] < 0 || beta[n] >= b || kvhead[n] < 0 || kvhead[n] >= Hkl ||
        key[n] < 0 || key[n] >= S)
      return ORC_ERR_RANGE;
  long n_rep = Hl / Hkl;
#pragma omp parallel for schedule(dynamic, 1)
  for (long n = 0; n < nsamp; ++n) {
    long bt = beta[n], kvh = kvhead[n], j = key[n];
    const double *kj = k + ((bt * S + j) * Hkl + kvh) * d;
    const double *vj = v + ((bt * S + j) * Hkl + kvh) * d;
    double *dkj = dk_out + n * d, *dvj = dv_out + n * d;
    for (long e = 0; e < d; ++e) dkj[e] = dvj[e] = 0.0;
    for (long h = kvh * n_rep; h < (kvh + 1) * n_rep; ++h)
      for (long i = j; i < S; ++i) {
        const double *qi = q + ((bt * S + i) * Hl + h) * d;
        const double *doi = dout + ((bt * S + i) * Hl + h) * d;
        const double *oi = o + ((bt * S + i) * Hl + h) * d;
        double Di = dot(doi, oi, d);
        double p = exp(scale * dot(qi, kj, d) - lse[(bt * Hl + h) * S + i]);
        double ds = p * (dot(doi, vj, d) - Di);
        for (long e = 0; e < d; ++e) {
          dvj[e] += p * doi[e];
          dkj[e] += scale * ds * qi[e];
        }
      }
  }
  return ORC_OK;
}

int oracle_attn_rows(const double *q, const double *k, const double *v,
                     const double *dout, long b, long S, long Hl, long Hkl,
                     long d, double scale, long nsamp, const long *beta,
                     const long *head, const long *row, double *o_out,
                     double *lse_out, double *dq_out) {
  int rc = attn_args_ok(b, S, Hl, Hkl, d);
  if (rc) return rc;
  if (nsamp < 0) return ORC_ERR_RANGE;
  if (!q || !k || !v || !dout || !beta || !head || !row || !o_out ||
      !lse_out || !dq_out)
    return ORC_ERR_NULL;
  for (long n = 0; n < nsamp; ++n)
    if (beta[n] < 0 || beta[n] >= b || head[n] < 0 || head[n] >= Hl ||
        row[n] < 0 || row[n] >= S)
      return ORC_ERR_RANGE;
  long n_rep = Hl / Hkl;
#pragma omp parallel
  {
    double *s = (double *)malloc(sizeof(double) * (size_t)(S > 0 ? S : 1));
#pragma omp for schedule(dynamic, 1)
    for (long n = 0; n < nsamp; ++n) {
      long bt = beta[n], h = head[n], i = row[n], kvh = h / n_rep;
      double *oi = o_out + n * d;
      double Li = fwd_row(q, k, v, oi, s, S, Hl, Hkl, d, scale, bt, h, i);
      lse_out[n] = Li;
      const double *qi = q + ((bt * S + i) * Hl + h) * d;
      const double *doi = dout + ((bt * S + i) * Hl + h) * d;
      double Di = dot(doi, oi, d);
      double *dqi = dq_out + n * d;
      for (long e = 0; e < d; ++e) dqi[e] = 0.0;
      for (long j = 0; j <= i; ++j) {
        const double *kj = k + ((bt * S + j) * Hkl + kvh) * d;
        const double *vj = v + ((bt * S + j) * Hkl + kvh) * d;
        double p = exp(scale * dot(qi, kj, d) - Li);
        double ds = p * (dot(doi, vj, d) - Di);
        for (long e = 0; e < d; ++e) dqi[e] += scale * ds * kj[e];
      }
    }
    free(s);
  }
  return ORC_OK;
}
