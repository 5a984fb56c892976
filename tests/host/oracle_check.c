/* Host run of every oracle function on small shapes, meant to be built with
 * AddressSanitizer and UndefinedBehaviorSanitizer: argument errors, the
 * permutations (pack after unpack and the exchange's send/receive sides are
 * identities, a shared head is added and summed), attention forward and
 * backward with ragged sizes and GQA, and the row and key samples against the
 * full computation.  Prints "oracle ok <checks>"; exits 1 at the first
 * failure. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../oracle/basp_oracle.h"

static int checks = 0;
#define CHECK(c)                                           \
  do {                                                     \
    ++checks;                                              \
    if (!(c)) {                                            \
      printf("FAIL line %d: %s\n", __LINE__, #c);          \
      return 1;                                            \
    }                                                      \
  } while (0)

static unsigned long long rng = 0x243F6A8885A308D3ull;
static double urand(void) { /* xorshift64*, uniform in [-1, 1) */
  rng ^= rng >> 12;
  rng ^= rng << 25;
  rng ^= rng >> 27;
  return (double)((rng * 0x2545F4914F6CDD1Dull) >> 11) / (double)(1ull << 52) - 1.0;
}

static int permutations(void) {
  enum { b = 2, S = 24, n = 6, d = 5, G = 3, Sg = S / G };
  unsigned short *sh[G], *back[G];
  for (int j = 0; j < G; ++j) {
    sh[j] = malloc(sizeof(unsigned short) * b * Sg * n * d);
    back[j] = calloc(b * Sg * n * d, sizeof(unsigned short));
    for (int i = 0; i < b * Sg * n * d; ++i) sh[j][i] = (unsigned short)(rng = rng * 6364136223846793005ull + j + 1);
  }
  unsigned short *loc = malloc(sizeof(unsigned short) * b * S * (n / G) * d);
  for (int r = 0; r < G; ++r) {
    CHECK(oracle_pack((const void *const *)sh, loc, b, S, n, d, G, r, 2) == 0);
    CHECK(oracle_unpack(loc, (void *const *)back, b, S, n, d, G, r, 2) == 0);
  }
  for (int j = 0; j < G; ++j) CHECK(memcmp(sh[j], back[j], sizeof(unsigned short) * b * Sg * n * d) == 0);
  /* the owner's side: send blocks, then receive them back */
  unsigned short *send = malloc(sizeof(unsigned short) * G * b * Sg * (n / G) * d);
  unsigned short *own = malloc(sizeof(unsigned short) * b * Sg * n * d);
  CHECK(oracle_a2a_pack(sh[1], send, b, S, n, d, G, 2) == 0);
  CHECK(oracle_a2a_unpack(send, own, b, S, n, d, G, 2) == 0);
  CHECK(memcmp(own, sh[1], sizeof(unsigned short) * b * Sg * n * d) == 0);
  /* errors */
  CHECK(oracle_pack((const void *const *)sh, loc, b, S + 1, n, d, G, 0, 2) < 0);
  CHECK(oracle_pack((const void *const *)sh, loc, b, S, n, d, G, G, 2) < 0);
  CHECK(oracle_pack((const void *const *)sh, loc, b, S, n, d, G, 0, 3) < 0);
  CHECK(oracle_pack(NULL, loc, b, S, n, d, G, 0, 2) < 0);
  CHECK(oracle_unpack(loc, NULL, b, S, n, d, G, 0, 2) < 0);
  CHECK(oracle_a2a_pack(NULL, send, b, S, n, d, G, 2) < 0);
  CHECK(oracle_pack((const void *const *)sh, loc, 0, S, n, d, G, 0, 2) == 0);
  for (int j = 0; j < G; ++j) {
    free(sh[j]);
    free(back[j]);
  }
  free(loc);
  free(send);
  free(own);

  /* a shared head (n = 2 heads, G = 4 members): add and sum in fp32 */
  enum { G4 = 4, n2 = 2, S4 = 8, Sg4 = S4 / G4 };
  float *dsh[G4];
  for (int j = 0; j < G4; ++j) dsh[j] = calloc(1 * Sg4 * n2 * d, sizeof(float));
  float *part = malloc(sizeof(float) * S4 * d);
  for (int i = 0; i < S4 * d; ++i) part[i] = (float)(i % 7);
  for (int r = 0; r < G4; ++r) CHECK(oracle_unpack_add(part, dsh, 1, S4, n2, d, G4, r) == 0);
  /* head h of shard j: the sum of the G/n = 2 members sharing it */
  for (int j = 0; j < G4; ++j)
    for (int t = 0; t < Sg4; ++t)
      for (int h = 0; h < n2; ++h)
        for (int e = 0; e < d; ++e)
          CHECK(dsh[j][(t * n2 + h) * d + e] == 2.0f * part[((j * Sg4 + t)) * d + e]);
  float *recv = malloc(sizeof(float) * G4 * Sg4 * d), *own4 = malloc(sizeof(float) * Sg4 * n2 * d);
  for (int i = 0; i < G4 * Sg4 * d; ++i) recv[i] = (float)(i % 5);
  CHECK(oracle_a2a_unpack(recv, own4, 1, S4, n2, d, G4, 4) == 0);
  for (int t = 0; t < Sg4; ++t)
    for (int h = 0; h < n2; ++h)
      for (int e = 0; e < d; ++e)
        CHECK(own4[(t * n2 + h) * d + e] ==
              recv[((2 * h) * Sg4 + t) * d + e] + recv[((2 * h + 1) * Sg4 + t) * d + e]);
  CHECK(oracle_a2a_unpack(recv, own4, 1, S4, n2, d, G4, 2) < 0); /* bf16 sum refused */
  for (int j = 0; j < G4; ++j) free(dsh[j]);
  free(part);
  free(recv);
  free(own4);
  return 0;
}

static int attention(void) {
  enum { b = 2, S = 19, Hl = 4, Hkl = 2, d = 6 };
  const double c = 0.4;
  const size_t nq = (size_t)b * S * Hl * d, nk = (size_t)b * S * Hkl * d;
  double *q = malloc(nq * 8), *k = malloc(nk * 8), *v = malloc(nk * 8), *dout = malloc(nq * 8);
  for (size_t i = 0; i < nq; ++i) q[i] = urand(), dout[i] = urand();
  for (size_t i = 0; i < nk; ++i) k[i] = urand(), v[i] = urand();
  double *o = malloc(nq * 8), *lse = malloc((size_t)b * Hl * S * 8);
  CHECK(oracle_attn_fwd(q, k, v, o, lse, b, S, Hl, Hkl, d, c, 0, S) == 0);
  for (int bt = 0; bt < b; ++bt)
    for (int h = 0; h < Hl; ++h)
      for (int e = 0; e < d; ++e)
        CHECK(o[((bt * S) * Hl + h) * d + e] == v[((bt * S) * Hkl + h / 2) * d + e]);
  double *dq = malloc(nq * 8), *dk = malloc(nk * 8), *dv = malloc(nk * 8);
  CHECK(oracle_attn_bwd(q, k, v, dout, o, lse, dq, dk, dv, b, S, Hl, Hkl, d, c, 0) == 0);
  /* sum_j dK_j = 0 per (sequence, kv head, column) */
  for (int bt = 0; bt < b; ++bt)
    for (int g = 0; g < Hkl; ++g)
      for (int e = 0; e < d; ++e) {
        double s = 0.0;
        for (int j = 0; j < S; ++j) s += dk[((bt * S + j) * Hkl + g) * d + e];
        CHECK(fabs(s) < 1e-12);
      }
  /* rows [7, S) alone */
  const int r0 = 7, R = S - r0;
  double *o2 = malloc((size_t)b * R * Hl * d * 8), *l2 = malloc((size_t)b * Hl * R * 8);
  CHECK(oracle_attn_fwd(q, k, v, o2, l2, b, S, Hl, Hkl, d, c, r0, S) == 0);
  double *dq2 = malloc((size_t)b * R * Hl * d * 8), *dk2 = malloc((size_t)b * R * Hkl * d * 8),
         *dv2 = malloc((size_t)b * R * Hkl * d * 8);
  CHECK(oracle_attn_bwd(q, k, v, dout, o2, l2, dq2, dk2, dv2, b, S, Hl, Hkl, d, c, r0) == 0);
  for (int bt = 0; bt < b; ++bt)
    for (int r = 0; r < R; ++r)
      for (int g = 0; g < Hkl; ++g)
        for (int e = 0; e < d; ++e)
          CHECK(fabs(dk2[((bt * R + r) * Hkl + g) * d + e] -
                     dk[((bt * S + r0 + r) * Hkl + g) * d + e]) < 1e-13);
  /* row and key samples */
  long beta[3] = {0, 1, 1}, head[3] = {3, 0, 2}, row[3] = {0, S - 1, 9};
  double os[3 * d], ls[3], dqs[3 * d];
  CHECK(oracle_attn_rows(q, k, v, dout, b, S, Hl, Hkl, d, c, 3, beta, head, row, os, ls, dqs) == 0);
  for (int n = 0; n < 3; ++n) {
    CHECK(fabs(ls[n] - lse[(beta[n] * Hl + head[n]) * S + row[n]]) < 1e-13);
    for (int e = 0; e < d; ++e)
      CHECK(fabs(dqs[n * d + e] - dq[((beta[n] * S + row[n]) * Hl + head[n]) * d + e]) < 1e-13);
  }
  long kvh[3] = {1, 0, 1}, key[3] = {0, S - 1, 5};
  double dks[3 * d], dvs[3 * d];
  CHECK(oracle_attn_keys(q, k, v, dout, o, lse, b, S, Hl, Hkl, d, c, 3, beta, kvh, key, dks, dvs) == 0);
  for (int n = 0; n < 3; ++n)
    for (int e = 0; e < d; ++e) {
      CHECK(fabs(dks[n * d + e] - dk[((beta[n] * S + key[n]) * Hkl + kvh[n]) * d + e]) < 1e-13);
      CHECK(fabs(dvs[n * d + e] - dv[((beta[n] * S + key[n]) * Hkl + kvh[n]) * d + e]) < 1e-13);
    }
  /* errors */
  long bad[1] = {S};
  CHECK(oracle_attn_keys(q, k, v, dout, o, lse, b, S, Hl, Hkl, d, c, 1, beta, kvh, bad, dks, dvs) < 0);
  CHECK(oracle_attn_rows(q, k, v, dout, b, S, Hl, Hkl, d, c, 1, beta, head, bad, os, ls, dqs) < 0);
  CHECK(oracle_attn_fwd(q, k, v, o, lse, b, S, Hl, 3, d, c, 0, S) < 0);
  CHECK(oracle_attn_fwd(q, k, v, o, lse, b, S, Hl, Hkl, d, c, 5, 4) < 0);
  CHECK(oracle_attn_bwd(q, k, v, dout, o, lse, dq, dk, dv, b, S, Hl, Hkl, d, c, S + 1) < 0);
  CHECK(oracle_attn_fwd(NULL, k, v, o, lse, b, S, Hl, Hkl, d, c, 0, S) < 0);
  CHECK(oracle_attn_fwd(q, k, v, o, lse, 0, S, Hl, Hkl, d, c, 0, S) == 0);
  free(q), free(k), free(v), free(dout), free(o), free(lse), free(dq), free(dk), free(dv);
  free(o2), free(l2), free(dq2), free(dk2), free(dv2);
  return 0;
}

int main(void) {
  long g, l, K, s0, s1, t0, t1;
  CHECK(oracle_group_of(4, 2, 3, &g, &l, &K) == 0 && g == 1 && l == 1 && K == 2);
  CHECK(oracle_group_of(4, 8, 0, &g, &l, &K) < 0);
  CHECK(oracle_seq_partition(16384, 4, 6, &s0, &s1, &t0, &t1) == 0 && s0 == 1 && t0 == 8192);
  CHECK(oracle_seq_partition(10, 4, 0, &s0, &s1, &t0, &t1) < 0);
  oracle_set_threads(2);
  CHECK(oracle_threads() == 2);
  if (permutations()) return 1;
  if (attention()) return 1;
  oracle_set_threads(1);
  if (permutations()) return 1;
  if (attention()) return 1;
  printf("oracle ok %d\n", checks);
  return 0;
}
