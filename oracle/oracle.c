/*
 * oracle.c -- plain fp64 CPU implementation of the batched cGRU-attention
 * decoder step (the paper's Section 5.1 forward step NMT(H_{i-1}, E_i)),
 * plus the source-side initialisation it assumes (precomputed source
 * context, Section 5.1 opening paragraph).
 *
 * TEST INFRASTRUCTURE ONLY: slow, obviously correct, and independent of the
 * HIP library.  Equations and readings are listed in oracle.h.
 *
 * ORACLE_PLANT_<NAME> compile switches each plant one deliberate mistake
 * (RESET, ZSWAP, BWDORDER, WQT, NOMASK, G2BIAS, READOUT_S1, LSEDROP); the
 * pin tests build these variants to show that some pin fails for each.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double sigmoid(double x) { return 1.0 / (1.0 + exp(-x)); }

int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* y[j] += sum_k x[k] * W[k][j] for a row vector x [nin] and W [nin x ncol]. */
static void vec_mat_acc(int nin, int ncol, const double* x, const float* W, double* y) {
  for (int k = 0; k < nin; ++k) {
    double xk = x[k];
    const float* row = W + (size_t)k * ncol;
    for (int j = 0; j < ncol; ++j) y[j] += xk * (double)row[j];
  }
}

/* One GRU cell for a single row: the DL4MT form with the reset gate applied
 * after the state-side product (r * (h Un + bs_n)). */
static void gru_row(int nin, int H, const double* u, const double* h, const float* W,
                    const float* U, const float* b_in, const float* b_st, double* out,
                    double* gi, double* gh) {
  int G = 3 * H;
  for (int j = 0; j < G; ++j) {
    gi[j] = b_in ? (double)b_in[j] : 0.0;
    gh[j] = b_st ? (double)b_st[j] : 0.0;
  }
  if (u) vec_mat_acc(nin, G, u, W, gi);
  vec_mat_acc(H, G, h, U, gh);
  for (int j = 0; j < H; ++j) {
    double r = sigmoid(gi[j] + gh[j]);
    double z = sigmoid(gi[H + j] + gh[H + j]);
#ifdef ORACLE_PLANT_RESET
    r = 1.0; /* planted: reset gate dropped */
#endif
    double n = tanh(gi[2 * H + j] + r * gh[2 * H + j]);
#ifdef ORACLE_PLANT_ZSWAP
    out[j] = (1.0 - z) * h[j] + z * n; /* planted: update gate roles swapped */
#else
    out[j] = z * h[j] + (1.0 - z) * n;
#endif
  }
}

int oracle_gru(int32_t n, int32_t nin, int32_t H, const double* u, const double* h,
               const float* W, const float* U, const float* b_in, const float* b_st,
               double* h_out) {
  if (n < 0 || nin < 0 || H <= 0 || !h || !U || !h_out || (nin > 0 && (!u || !W)))
    return ORACLE_EINVAL;
#pragma omp parallel
  {
    double* gi = (double*)malloc(sizeof(double) * 3 * H);
    double* gh = (double*)malloc(sizeof(double) * 3 * H);
#pragma omp for schedule(static)
    for (int b = 0; b < n; ++b)
      gru_row(nin, H, nin ? u + (size_t)b * nin : NULL, h + (size_t)b * H, W, U, b_in, b_st,
              h_out + (size_t)b * H, gi, gh);
    free(gi);
    free(gh);
  }
  return ORACLE_OK;
}

static int check_dims(const oracle_dims* d) {
  return d && d->V > 0 && d->V_src > 0 && d->E > 0 && d->H > 0 && d->A > 0;
}

/* Attention keys and initial state from annotations of one sentence. */
static void keys_and_init(const oracle_dims* d, const oracle_weights* w, int Tpad, int L,
                          const double* ctx_s, double* pctx_s, double* s0_s) {
  int H = d->H, A = d->A, C = 2 * d->H;
  if (pctx_s) {
    for (int i = 0; i < Tpad; ++i) {
      double* p = pctx_s + (size_t)i * A;
      if (i >= L) {
        memset(p, 0, sizeof(double) * A);
        continue;
      }
      for (int a = 0; a < A; ++a) p[a] = (double)w->att_b[a];
      vec_mat_acc(C, A, ctx_s + (size_t)i * C, w->att_Wc, p);
    }
  }
  if (s0_s) {
    double* mean = (double*)calloc(C, sizeof(double));
    for (int i = 0; i < L; ++i)
      for (int k = 0; k < C; ++k) mean[k] += ctx_s[(size_t)i * C + k];
    for (int k = 0; k < C; ++k) mean[k] /= (double)L;
    for (int j = 0; j < H; ++j) s0_s[j] = (double)w->init_b[j];
    vec_mat_acc(C, H, mean, w->init_W, s0_s);
    for (int j = 0; j < H; ++j) s0_s[j] = tanh(s0_s[j]);
    free(mean);
  }
}

int oracle_encode(const oracle_dims* d, const oracle_weights* w, int32_t S, int32_t Tpad,
                  const int32_t* src_ids, const int32_t* len, double* ctx, double* pctx,
                  double* s0) {
  if (!check_dims(d) || !w || S < 0 || Tpad <= 0 || !src_ids || !len) return ORACLE_EINVAL;
  for (int s = 0; s < S; ++s) {
    if (len[s] < 1 || len[s] > Tpad) return ORACLE_EINVAL;
    for (int i = 0; i < len[s]; ++i)
      if (src_ids[(size_t)s * Tpad + i] < 0 || src_ids[(size_t)s * Tpad + i] >= d->V_src)
        return ORACLE_ERANGE;
  }
  int E = d->E, H = d->H, A = d->A, C = 2 * d->H;
  int status = ORACLE_OK;
  double* ctx_all = ctx ? ctx : (double*)malloc(sizeof(double) * (size_t)S * Tpad * C);
#pragma omp parallel
  {
    double* x = (double*)malloc(sizeof(double) * E);
    double* h = (double*)malloc(sizeof(double) * H);
    double* hn = (double*)malloc(sizeof(double) * H);
    double* gi = (double*)malloc(sizeof(double) * 3 * H);
    double* gh = (double*)malloc(sizeof(double) * 3 * H);
#pragma omp for schedule(dynamic, 1)
    for (int s = 0; s < S; ++s) {
      int L = len[s];
      double* cs = ctx_all + (size_t)s * Tpad * C;
      memset(cs, 0, sizeof(double) * (size_t)Tpad * C);
      /* forward direction over positions 0..L-1 */
      for (int j = 0; j < H; ++j) h[j] = 0.0;
      for (int i = 0; i < L; ++i) {
        const float* e = w->emb_src + (size_t)src_ids[(size_t)s * Tpad + i] * E;
        for (int k = 0; k < E; ++k) x[k] = (double)e[k];
        gru_row(E, H, x, h, w->enc_f_W, w->enc_f_U, w->enc_f_b, NULL, hn, gi, gh);
        memcpy(h, hn, sizeof(double) * H);
        memcpy(cs + (size_t)i * C, h, sizeof(double) * H);
      }
      /* backward direction over positions L-1..0 */
      for (int j = 0; j < H; ++j) h[j] = 0.0;
#ifdef ORACLE_PLANT_BWDORDER
      for (int i = 0; i < L; ++i) { /* planted: backward pass run left to right */
#else
      for (int i = L - 1; i >= 0; --i) {
#endif
        const float* e = w->emb_src + (size_t)src_ids[(size_t)s * Tpad + i] * E;
        for (int k = 0; k < E; ++k) x[k] = (double)e[k];
        gru_row(E, H, x, h, w->enc_b_W, w->enc_b_U, w->enc_b_b, NULL, hn, gi, gh);
        memcpy(h, hn, sizeof(double) * H);
        memcpy(cs + (size_t)i * C + H, h, sizeof(double) * H);
      }
      keys_and_init(d, w, Tpad, L, cs, pctx ? pctx + (size_t)s * Tpad * A : NULL,
                    s0 ? s0 + (size_t)s * H : NULL);
    }
    free(x);
    free(h);
    free(hn);
    free(gi);
    free(gh);
  }
  if (!ctx) free(ctx_all);
  return status;
}

int oracle_keys_from_annotations(const oracle_dims* d, const oracle_weights* w, int32_t S,
                                 int32_t Tpad, const float* ctx_f32, const int32_t* len,
                                 double* ctx, double* pctx) {
  if (!check_dims(d) || !w || S < 0 || Tpad <= 0 || !ctx_f32 || !len || !ctx) return ORACLE_EINVAL;
  for (int s = 0; s < S; ++s)
    if (len[s] < 1 || len[s] > Tpad) return ORACLE_EINVAL;
  int A = d->A, C = 2 * d->H;
  for (int s = 0; s < S; ++s)
    for (int i = 0; i < Tpad; ++i)
      for (int k = 0; k < C; ++k) {
        size_t o = ((size_t)s * Tpad + i) * C + k;
        ctx[o] = i < len[s] ? (double)ctx_f32[o] : 0.0;
      }
#pragma omp parallel for schedule(dynamic, 1)
  for (int s = 0; s < S; ++s)
    keys_and_init(d, w, Tpad, len[s], ctx + (size_t)s * Tpad * C,
                  pctx ? pctx + (size_t)s * Tpad * A : NULL, NULL);
  return ORACLE_OK;
}

/* Log-sum-exp over one row of logits, shifted by the maximum. */
static double log_sum_exp(int V, const double* z) {
  double m = z[0];
  for (int v = 1; v < V; ++v)
    if (z[v] > m) m = z[v];
  double s = 0.0;
#ifdef ORACLE_PLANT_LSEDROP
  V -= 1; /* planted: last vocabulary entry left out of the normaliser */
#endif
  for (int v = 0; v < V; ++v) s += exp(z[v] - m);
  return m + log(s);
}

static void logits_row(int E, int V, const double* t, const float* out_W, const float* out_b,
                       double* z) {
  for (int v = 0; v < V; ++v) z[v] = (double)out_b[v];
  vec_mat_acc(E, V, t, out_W, z);
}

int oracle_vocab_logsoftmax(int32_t B, int32_t E, int32_t V, const double* t,
                            const float* out_W, const float* out_b, const int32_t* req,
                            double* logp, double* logZ, double* logp_all) {
  if (B < 0 || E <= 0 || V <= 0 || !t || !out_W || !out_b) return ORACLE_EINVAL;
  if (req)
    for (int b = 0; b < B; ++b)
      if (req[b] < 0 || req[b] >= V) return ORACLE_ERANGE;
#pragma omp parallel
  {
    double* z = (double*)malloc(sizeof(double) * V);
#pragma omp for schedule(dynamic, 1)
    for (int b = 0; b < B; ++b) {
      logits_row(E, V, t + (size_t)b * E, out_W, out_b, z);
      double lz = log_sum_exp(V, z);
      if (logZ) logZ[b] = lz;
      if (logp && req) logp[b] = z[req[b]] - lz;
      if (logp_all)
        for (int v = 0; v < V; ++v) logp_all[(size_t)b * V + v] = z[v] - lz;
    }
    free(z);
  }
  return ORACLE_OK;
}

/* The decoder step for one row.  Scratch: gi, gh [3H]; x [E]; s1 [H];
 * q [A]; e [Tpad]; c [C]; s2 [H]; t [E]; z [V]. */
typedef struct {
  double *gi, *gh, *x, *s1, *q, *e, *c, *s2, *t, *z;
} row_scratch;

static void score_row(const oracle_dims* d, const oracle_weights* w, int Tpad,
                      const double* ctx_s, const double* pctx_s, int L, const double* s_prev,
                      int y_prev, int req, row_scratch* r, double* logp, double* s_new,
                      double* logZ, double* alpha, double* c_out, double* s1_out,
                      double* t_out) {
  int E = d->E, H = d->H, A = d->A, V = d->V, C = 2 * d->H;
  /* previous-word embedding; the sentence start uses the zero vector */
  for (int k = 0; k < E; ++k) r->x[k] = y_prev >= 0 ? (double)w->emb_tgt[(size_t)y_prev * E + k] : 0.0;
  /* first GRU: input-side bias, no state-side bias */
  gru_row(E, H, r->x, s_prev, w->g1_W, w->g1_U, w->g1_b, NULL, r->s1, r->gi, r->gh);
  /* MLP attention over the unmasked source positions */
  for (int a = 0; a < A; ++a) r->q[a] = 0.0;
#ifdef ORACLE_PLANT_WQT
  for (int a = 0; a < A; ++a) /* planted: query weights read transposed (needs H == A) */
    for (int k = 0; k < H; ++k) r->q[a] += r->s1[k] * (double)w->att_Wq[(size_t)a * H + k];
#else
  vec_mat_acc(H, A, r->s1, w->att_Wq, r->q);
#endif
#ifdef ORACLE_PLANT_NOMASK
  L = Tpad; /* planted: attention ignores the source length */
#endif
  double emax = -INFINITY;
  for (int i = 0; i < L; ++i) {
    const double* p = pctx_s + (size_t)i * A;
    double e = 0.0;
    for (int a = 0; a < A; ++a) e += (double)w->att_v[a] * tanh(p[a] + r->q[a]);
    r->e[i] = e;
    if (e > emax) emax = e;
  }
  double esum = 0.0;
  for (int i = 0; i < L; ++i) {
    r->e[i] = exp(r->e[i] - emax);
    esum += r->e[i];
  }
  for (int i = 0; i < L; ++i) r->e[i] /= esum;
  for (int i = L; i < Tpad; ++i) r->e[i] = 0.0;
  for (int k = 0; k < C; ++k) r->c[k] = 0.0;
  for (int i = 0; i < L; ++i)
    for (int k = 0; k < C; ++k) r->c[k] += r->e[i] * ctx_s[(size_t)i * C + k];
  /* second GRU: context as input, state-side bias inside the reset gate */
#ifdef ORACLE_PLANT_G2BIAS
  gru_row(C, H, r->c, r->s1, w->g2_Wc, w->g2_U, w->g2_b, NULL, r->s2, r->gi, r->gh); /* planted */
#else
  gru_row(C, H, r->c, r->s1, w->g2_Wc, w->g2_U, NULL, w->g2_b, r->s2, r->gi, r->gh);
#endif
  /* tanh readout from the new state, the previous word and the context */
  for (int k = 0; k < E; ++k) r->t[k] = (double)w->ro_b[k];
#ifdef ORACLE_PLANT_READOUT_S1
  vec_mat_acc(H, E, r->s1, w->ro_Ws, r->t); /* planted: readout from the first-GRU state */
#else
  vec_mat_acc(H, E, r->s2, w->ro_Ws, r->t);
#endif
  vec_mat_acc(E, E, r->x, w->ro_Wy, r->t);
  vec_mat_acc(C, E, r->c, w->ro_Wc, r->t);
  for (int k = 0; k < E; ++k) r->t[k] = tanh(r->t[k]);
  /* full-vocabulary log-softmax and the requested word */
  logits_row(E, V, r->t, w->out_W, w->out_b, r->z);
  double lz = log_sum_exp(V, r->z);
  if (logp) *logp = r->z[req] - lz;
  if (logZ) *logZ = lz;
  if (s_new) memcpy(s_new, r->s2, sizeof(double) * H);
  if (alpha) memcpy(alpha, r->e, sizeof(double) * Tpad);
  if (c_out) memcpy(c_out, r->c, sizeof(double) * C);
  if (s1_out) memcpy(s1_out, r->s1, sizeof(double) * H);
  if (t_out) memcpy(t_out, r->t, sizeof(double) * E);
}

static int score_impl(const oracle_dims* d, const oracle_weights* w, int32_t S, int32_t Tpad,
                      const double* ctx, const double* pctx, const int32_t* len, int32_t B,
                      const float* s_prev_f, const double* s_prev_d, const int32_t* y_prev,
                      const int32_t* sent_id, const int32_t* req, double* logp, double* s_new,
                      double* logZ, double* alpha, double* c, double* s1, double* t) {
  if (!check_dims(d) || !w || S <= 0 || Tpad <= 0 || B < 0 || !ctx || !pctx || !len ||
      !y_prev || !sent_id || !req || (!s_prev_f && !s_prev_d))
    return ORACLE_EINVAL;
  for (int s = 0; s < S; ++s)
    if (len[s] < 1 || len[s] > Tpad) return ORACLE_EINVAL;
  for (int b = 0; b < B; ++b)
    if (y_prev[b] < -1 || y_prev[b] >= d->V || req[b] < 0 || req[b] >= d->V || sent_id[b] < 0 ||
        sent_id[b] >= S)
      return ORACLE_ERANGE;
  int E = d->E, H = d->H, A = d->A, V = d->V, C = 2 * d->H;
#pragma omp parallel
  {
    row_scratch r;
    r.gi = (double*)malloc(sizeof(double) * 3 * H);
    r.gh = (double*)malloc(sizeof(double) * 3 * H);
    r.x = (double*)malloc(sizeof(double) * E);
    r.s1 = (double*)malloc(sizeof(double) * H);
    r.q = (double*)malloc(sizeof(double) * A);
    r.e = (double*)malloc(sizeof(double) * Tpad);
    r.c = (double*)malloc(sizeof(double) * C);
    r.s2 = (double*)malloc(sizeof(double) * H);
    r.t = (double*)malloc(sizeof(double) * E);
    r.z = (double*)malloc(sizeof(double) * V);
    double* sp = (double*)malloc(sizeof(double) * H);
#pragma omp for schedule(dynamic, 1)
    for (int b = 0; b < B; ++b) {
      int s = sent_id[b];
      for (int j = 0; j < H; ++j)
        sp[j] = s_prev_d ? s_prev_d[(size_t)b * H + j] : (double)s_prev_f[(size_t)b * H + j];
      score_row(d, w, Tpad, ctx + (size_t)s * Tpad * C, pctx + (size_t)s * Tpad * A, len[s], sp,
                y_prev[b], req[b], &r, logp ? logp + b : NULL,
                s_new ? s_new + (size_t)b * H : NULL, logZ ? logZ + b : NULL,
                alpha ? alpha + (size_t)b * Tpad : NULL, c ? c + (size_t)b * C : NULL,
                s1 ? s1 + (size_t)b * H : NULL, t ? t + (size_t)b * E : NULL);
    }
    free(r.gi);
    free(r.gh);
    free(r.x);
    free(r.s1);
    free(r.q);
    free(r.e);
    free(r.c);
    free(r.s2);
    free(r.t);
    free(r.z);
    free(sp);
  }
  return ORACLE_OK;
}

int oracle_score_batch(const oracle_dims* d, const oracle_weights* w, int32_t S, int32_t Tpad,
                       const double* ctx, const double* pctx, const int32_t* len, int32_t B,
                       const float* s_prev, const int32_t* y_prev, const int32_t* sent_id,
                       const int32_t* req, double* logp, double* s_new, double* logZ,
                       double* alpha, double* c, double* s1, double* t) {
  return score_impl(d, w, S, Tpad, ctx, pctx, len, B, s_prev, NULL, y_prev, sent_id, req, logp,
                    s_new, logZ, alpha, c, s1, t);
}

int oracle_score_batch_f64state(const oracle_dims* d, const oracle_weights* w, int32_t S,
                                int32_t Tpad, const double* ctx, const double* pctx,
                                const int32_t* len, int32_t B, const double* s_prev,
                                const int32_t* y_prev, const int32_t* sent_id,
                                const int32_t* req, double* logp, double* s_new, double* logZ,
                                double* alpha, double* c, double* s1, double* t) {
  return score_impl(d, w, S, Tpad, ctx, pctx, len, B, NULL, s_prev, y_prev, sent_id, req, logp,
                    s_new, logZ, alpha, c, s1, t);
}
