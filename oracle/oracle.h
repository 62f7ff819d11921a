/*
 * oracle.h -- fp64 CPU oracle for one batched step of the attentional
 * conditional-GRU decoder that the paper queries from phrase-based decoding.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or helper with the HIP library; the two meet only through
 * the seeded input arrays.
 *
 * The paper (Sections 1 and 3) names the model: the attentional
 * encoder-decoder of Bahdanau et al. in its DL4MT / Nematus variant, with
 * embeddings of 500 and hidden layers of 1024.  Section 5.1 ("Scoring
 * hypotheses and their expansions") defines the query this oracle answers:
 * given the precomputed source context, one forward step maps a state
 * matrix and an embedding matrix (row-wise corresponding) to output states
 * and next-word probabilities.  The paper prints no equations; the readings
 * used here are the published DL4MT cGRU equations:
 *
 *   GRU(u, h): r = sig(u Wr + bi_r + h Ur + bs_r), z = sig(u Wz + bi_z + h Uz + bs_z)
 *              n = tanh(u Wn + bi_n + r * (h Un + bs_n)),  h' = z*h + (1-z)*n
 *   step:      x  = Emb[y_prev] (zero row for y_prev = -1)
 *              s1 = GRU(x, s_prev; g1_W, g1_U, bi = g1_b, bs = 0)
 *              e_i = v . tanh(pctx_i + s1 Wq),   alpha = softmax over i < L
 *              c  = sum_i alpha_i ctx_i
 *              s2 = GRU(c, s1; g2_Wc, g2_U, bi = 0, bs = g2_b)     (new state)
 *              t  = tanh(s2 Ws + x Wy + c Wc + b_r)
 *              z_v = t . out_W[:, v] + out_b[v],  logZ = log sum_v exp z_v
 *              logp = z_req - logZ
 *
 * Every computation is fp64 (inputs are fp32 and widened exactly); rows are
 * independent and run in an OpenMP loop.  No BLAS, no intrinsics.
 */
#ifndef NMT_ORACLE_H
#define NMT_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t V_src, V, E, H, A; /* C = 2H */
} oracle_dims;

/* Host fp32 parameters, x.W orientation ([in x out], row-major); the
 * 3H-wide GRU blocks are ordered [r | z | n]. */
typedef struct {
  const float *emb_src, *enc_f_W, *enc_f_b, *enc_f_U, *enc_b_W, *enc_b_b, *enc_b_U;
  const float *att_Wc, *att_b, *init_W, *init_b;
  const float *emb_tgt, *g1_W, *g1_b, *g1_U, *att_Wq, *att_v;
  const float *g2_U, *g2_b, *g2_Wc, *ro_Ws, *ro_Wy, *ro_Wc, *ro_b, *out_W, *out_b;
} oracle_weights;

/* Return codes. */
#define ORACLE_OK 0
#define ORACLE_EINVAL -1
#define ORACLE_ERANGE -4

/* One GRU cell for n rows (the reading above).  u [n x nin], h [n x H],
 * W [nin x 3H], U [H x 3H], b_in / b_st [3H] or NULL for zero.
 * Output h_out [n x H] (may not alias h). */
int oracle_gru(int32_t n, int32_t nin, int32_t H, const double* u, const double* h,
               const float* W, const float* U, const float* b_in, const float* b_st,
               double* h_out);

/* Bidirectional GRU encoder, attention keys and initial decoder state for
 * S sentences padded to Tpad.  src_ids [S x Tpad], len [S] (1..Tpad).
 * Outputs (any may be NULL): ctx [S x Tpad x 2H] (zero past each length),
 * pctx [S x Tpad x A] (zero past each length), s0 [S x H]. */
int oracle_encode(const oracle_dims* d, const oracle_weights* w, int32_t S, int32_t Tpad,
                  const int32_t* src_ids, const int32_t* len,
                  double* ctx, double* pctx, double* s0);

/* Attention keys from given annotations: pctx = ctx att_Wc + att_b for
 * i < len, zero past it.  ctx [S x Tpad x 2H] fp32. */
int oracle_keys_from_annotations(const oracle_dims* d, const oracle_weights* w, int32_t S,
                                 int32_t Tpad, const float* ctx_f32, const int32_t* len,
                                 double* ctx, double* pctx);

/* The batched decoder step.  ctx / pctx as produced above; s_prev [B x H]
 * fp32; y_prev [B] in [-1, V); sent_id [B] in [0, S); req [B] in [0, V).
 * Outputs (NULL = not wanted): logp [B], s_new [B x H], logZ [B],
 * alpha [B x Tpad], c [B x 2H], s1 [B x H], t [B x E]. */
int oracle_score_batch(const oracle_dims* d, const oracle_weights* w, int32_t S, int32_t Tpad,
                       const double* ctx, const double* pctx, const int32_t* len, int32_t B,
                       const float* s_prev, const int32_t* y_prev, const int32_t* sent_id,
                       const int32_t* req, double* logp, double* s_new, double* logZ,
                       double* alpha, double* c, double* s1, double* t);

/* Same step with the state given in fp64 (phrase scoring feeds s_new back). */
int oracle_score_batch_f64state(const oracle_dims* d, const oracle_weights* w, int32_t S,
                                int32_t Tpad, const double* ctx, const double* pctx,
                                const int32_t* len, int32_t B, const double* s_prev,
                                const int32_t* y_prev, const int32_t* sent_id,
                                const int32_t* req, double* logp, double* s_new, double* logZ,
                                double* alpha, double* c, double* s1, double* t);

/* Full-vocabulary log-softmax of the output layer for given readout
 * vectors t [B x E] (fp64): logZ [B] and logp of req [B] (req may be NULL).
 * logp_all [B x V] may be NULL. */
int oracle_vocab_logsoftmax(int32_t B, int32_t E, int32_t V, const double* t,
                            const float* out_W, const float* out_b, const int32_t* req,
                            double* logp, double* logZ, double* logp_all);

/* Number of OpenMP threads the oracle runs with. */
int oracle_num_threads(void);

#ifdef __cplusplus
}
#endif
#endif
