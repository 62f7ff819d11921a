/* Drives every entry point of the fp64 oracle (oracle/oracle.c) on small
 * random inputs under the address and undefined-behaviour sanitizers, with
 * the argument errors they must reject, and checks what the method fixes:
 * attention weights are a distribution over the unmasked positions, log
 * probabilities are at most 0 and a row's full distribution sums to 1. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>

#include "../../oracle/oracle.h"

#define CHECK(c)                                                   \
  do {                                                             \
    if (!(c)) {                                                    \
      fprintf(stderr, "check failed line %d: %s\n", __LINE__, #c); \
      exit(1);                                                     \
    }                                                              \
  } while (0)

static unsigned long long st = 88172645463325252ull;
static double urand(void) { /* xorshift64, uniform in [0, 1) */
  st ^= st << 13;
  st ^= st >> 7;
  st ^= st << 17;
  return (double)(st >> 11) / 9007199254740992.0;
}
static float* rnd(size_t n, double s) {
  float* a = (float*)malloc(sizeof(float) * (n ? n : 1));
  for (size_t i = 0; i < n; ++i) a[i] = (float)((2 * urand() - 1) * s);
  return a;
}

int main(void) {
  enum { Vs = 11, V = 13, E = 5, H = 6, A = 7, C = 2 * H, S = 3, T = 6, B = 9 };
  oracle_dims d = {Vs, V, E, H, A};
  oracle_weights w;
  w.emb_src = rnd((size_t)Vs * E, 0.5); w.enc_f_W = rnd((size_t)E * 3 * H, 0.5); w.enc_f_b = rnd(3 * H, 0.5);
  w.enc_f_U = rnd((size_t)H * 3 * H, 0.5); w.enc_b_W = rnd((size_t)E * 3 * H, 0.5); w.enc_b_b = rnd(3 * H, 0.5);
  w.enc_b_U = rnd((size_t)H * 3 * H, 0.5); w.att_Wc = rnd((size_t)C * A, 0.5); w.att_b = rnd(A, 0.5);
  w.init_W = rnd((size_t)C * H, 0.5); w.init_b = rnd(H, 0.5); w.emb_tgt = rnd((size_t)V * E, 0.5);
  w.g1_W = rnd((size_t)E * 3 * H, 0.5); w.g1_b = rnd(3 * H, 0.5); w.g1_U = rnd((size_t)H * 3 * H, 0.5);
  w.att_Wq = rnd((size_t)H * A, 0.5); w.att_v = rnd(A, 0.5); w.g2_U = rnd((size_t)H * 3 * H, 0.5);
  w.g2_b = rnd(3 * H, 0.5); w.g2_Wc = rnd((size_t)C * 3 * H, 0.5); w.ro_Ws = rnd((size_t)H * E, 0.5);
  w.ro_Wy = rnd((size_t)E * E, 0.5); w.ro_Wc = rnd((size_t)C * E, 0.5); w.ro_b = rnd(E, 0.5);
  w.out_W = rnd((size_t)E * V, 0.5); w.out_b = rnd(V, 0.5);
  int32_t ids[S * T], len[S] = {6, 1, 4};
  for (int i = 0; i < S * T; ++i) ids[i] = (int32_t)(urand() * Vs);
  double *ctx = calloc((size_t)S * T * C, 8), *pctx = calloc((size_t)S * T * A, 8), *s0 = calloc((size_t)S * H, 8);
  CHECK(oracle_encode(&d, &w, S, T, ids, len, ctx, pctx, s0) == ORACLE_OK);
  /* keys from given annotations */
  float* ann = rnd((size_t)S * T * C, 1.0);
  double *ctx2 = calloc((size_t)S * T * C, 8), *pctx2 = calloc((size_t)S * T * A, 8);
  CHECK(oracle_keys_from_annotations(&d, &w, S, T, ann, len, ctx2, pctx2) == ORACLE_OK);
  /* one step, fp32 and fp64 input states */
  float* sp = rnd((size_t)B * H, 0.9);
  double* spd = malloc(sizeof(double) * B * H);
  for (int i = 0; i < B * H; ++i) spd[i] = sp[i];
  int32_t y[B], sid[B], rq[B];
  for (int b = 0; b < B; ++b) {
    y[b] = b == 0 ? -1 : (int32_t)(urand() * V);
    sid[b] = (int32_t)(urand() * S);
    rq[b] = (int32_t)(urand() * V);
  }
  double logp[B], lz[B], *sn = malloc(8 * B * H), *al = malloc(8 * B * T), *c = malloc(8 * B * C),
                         *s1 = malloc(8 * B * H), *t = malloc(8 * B * E);
  CHECK(oracle_score_batch(&d, &w, S, T, ctx, pctx, len, B, sp, y, sid, rq, logp, sn, lz, al, c, s1, t) == ORACLE_OK);
  for (int b = 0; b < B; ++b) {
    double sum = 0;
    CHECK(logp[b] <= 0 && isfinite(lz[b]));
    for (int i = 0; i < T; ++i) {
      CHECK(al[b * T + i] >= 0);
      if (i >= len[sid[b]]) CHECK(al[b * T + i] == 0);
      sum += al[b * T + i];
    }
    CHECK(fabs(sum - 1) < 1e-12);
  }
  double logp2[B];
  CHECK(oracle_score_batch_f64state(&d, &w, S, T, ctx, pctx, len, B, spd, y, sid, rq, logp2, NULL, NULL, NULL, NULL,
                                    NULL, NULL) == ORACLE_OK);
  for (int b = 0; b < B; ++b) CHECK(logp2[b] == logp[b]);
  /* the full distribution of one readout sums to 1 */
  double all[V], lzr, lpr;
  int32_t r0 = 3;
  CHECK(oracle_vocab_logsoftmax(1, E, V, t, w.out_W, w.out_b, &r0, &lpr, &lzr, all) == ORACLE_OK);
  double tot = 0;
  for (int v = 0; v < V; ++v) tot += exp(all[v]);
  CHECK(fabs(tot - 1) < 1e-12 && lpr == all[3]);
  /* GRU cell on its own */
  double hout[2 * H];
  CHECK(oracle_gru(2, E, H, t, s1, w.g1_W, w.g1_U, w.g1_b, NULL, hout) == ORACLE_OK);
  /* argument errors */
  int32_t badlen[S] = {0, 1, 1}, badid[S * T];
  for (int i = 0; i < S * T; ++i) badid[i] = ids[i];
  badid[0] = Vs;
  CHECK(oracle_encode(&d, &w, S, T, ids, badlen, ctx, pctx, s0) != ORACLE_OK);
  CHECK(oracle_encode(&d, &w, S, T, badid, len, ctx, pctx, s0) != ORACLE_OK);
  int32_t bad_rq[B];
  for (int b = 0; b < B; ++b) bad_rq[b] = rq[b];
  bad_rq[B - 1] = V;
  CHECK(oracle_score_batch(&d, &w, S, T, ctx, pctx, len, B, sp, y, sid, bad_rq, logp, NULL, NULL, NULL, NULL, NULL,
                           NULL) != ORACLE_OK);
  CHECK(oracle_score_batch(NULL, &w, S, T, ctx, pctx, len, B, sp, y, sid, rq, logp, NULL, NULL, NULL, NULL, NULL,
                           NULL) != ORACLE_OK);
  printf("oracle driver ok\n");
  free(ctx); free(pctx); free(s0); free(ann); free(ctx2); free(pctx2); free(sp); free(spd);
  free(sn); free(al); free(c); free(s1); free(t);
  const float* const* fw = (const float* const*)&w;
  for (size_t i = 0; i < sizeof(w) / sizeof(float*); ++i) free((void*)fw[i]);
  return 0;
}
