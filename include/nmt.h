/*
 * nmt.h -- C-ABI of libnmt: batched querying of an attentional
 * conditional-GRU translation model from phrase-based decoding, on one
 * AMD Instinct MI355X (gfx950).
 *
 * The paper (Section 5.1, "Scoring hypotheses and their expansions";
 * Figure 2, procedure ScoreBatch) assumes the model has been initialised
 * with the source sentence, so that the source context is available at all
 * times, and then performs one forward step per tree depth:
 * (H_i, P_i) <- NMT(H_{i-1}, E_i), where the rows of the state matrix
 * H_{i-1} and of the embedding matrix E_i correspond one to one.  This
 * library exposes exactly those two operations:
 *
 *   nmt_encode       -- source initialisation: bidirectional GRU
 *                       annotations, attention keys and initial states.
 *   nmt_score_batch  -- one batched decoder step: new states H_i and the
 *                       normalised log-probability (natural log, full
 *                       vocabulary) of one requested next word per row.
 *                       The probability matrix P_i itself is never
 *                       materialised; only the requested entries and the
 *                       per-row log normaliser leave the device.
 *
 * Model (the DL4MT / Nematus variant of Bahdanau et al. named in Sections 1
 * and 3; C = 2H, gate blocks ordered [r | z | n], matrices in x.W
 * orientation [input dim x output dim], row-major):
 *   GRU(u, h; W, U, bi, bs):  r = sig(uW_r + bi_r + hU_r + bs_r)
 *                             z = sig(uW_z + bi_z + hU_z + bs_z)
 *                             n = tanh(uW_n + bi_n + r * (hU_n + bs_n))
 *                             h' = z*h + (1-z)*n
 *   encoder:  annotations ctx_i = [fwd GRU_i ; bwd GRU_i] (zero past the
 *             length), keys pctx_i = ctx_i att_Wc + att_b,
 *             s0 = tanh(mean_{i<L} ctx_i init_W + init_b)
 *   step:     x = emb_tgt[y_prev] (zero for y_prev = -1)
 *             s1 = GRU(x, s_prev; g1_W, g1_U, bi = g1_b, bs = 0)
 *             alpha = softmax_{i<L}( att_v . tanh(pctx_i + s1 att_Wq) )
 *             c = sum_i alpha_i ctx_i
 *             s_new = GRU(c, s1; g2_Wc, g2_U, bi = 0, bs = g2_b)
 *             t = tanh(s_new ro_Ws + x ro_Wy + c ro_Wc + ro_b)
 *             logZ = log sum_v exp(t out_W[:,v] + out_b[v])
 *             logp = t out_W[:,req] + out_b[req] - logZ
 *
 * Conventions for every call:
 *   - "d_" pointers are device memory owned by the caller (for example
 *     torch tensors passed by data_ptr()); "h_" pointers are host memory.
 *     fp32 device arrays must be 16-byte aligned.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Calls that
 *     take a stream enqueue work on it and return without waiting; host
 *     arguments are validated synchronously before anything is enqueued.
 *   - A non-OK status leaves nothing enqueued; nmt_last_error() returns a
 *     message for the calling thread.
 */
#ifndef NMT_H
#define NMT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct nmt_model nmt_model;   /* device copy of all weights (library-owned) */
typedef struct nmt_source nmt_source; /* ctx, pctx (and the factors e^{2 pctx} the score kernels
                                         read) and lengths of S sentences (library-owned) */

typedef enum {
  NMT_OK = 0,
  NMT_EINVAL = -1,     /* bad argument: null pointer, bad size, misaligned buffer */
  NMT_ENOMEM = -2,     /* device allocation failed */
  NMT_EDEVICE = -3,    /* HIP runtime error */
  NMT_ERANGE = -4,     /* an id was out of range (host-checked or reported by the device) */
  NMT_EWORKSPACE = -5  /* workspace smaller than nmt_score_workspace_bytes() */
} nmt_status;

typedef enum { NMT_F32 = 0, NMT_BF16 = 1 } nmt_dtype;

/* Model dimensions.  V_src / V: source / target vocabulary; E: embedding
 * width; H: hidden width (annotations are 2H wide); A: attention width.
 * E, H and A must be positive multiples of 4.  wtype selects the storage of
 * weights and embeddings on the device; activations, states and all
 * accumulation stay fp32. */
typedef struct {
  int32_t V_src, V, E, H, A;
  int32_t wtype; /* nmt_dtype */
} nmt_dims;

/* Host fp32 parameters (shapes with C = 2H):
 *   emb_src [V_src x E]; enc_f_W, enc_b_W [E x 3H]; enc_f_b, enc_b_b [3H];
 *   enc_f_U, enc_b_U [H x 3H]; att_Wc [C x A]; att_b [A]; init_W [C x H];
 *   init_b [H]; emb_tgt [V x E]; g1_W [E x 3H]; g1_b [3H]; g1_U [H x 3H];
 *   att_Wq [H x A]; att_v [A]; g2_U [H x 3H]; g2_b [3H]; g2_Wc [C x 3H];
 *   ro_Ws [H x E]; ro_Wy [E x E]; ro_Wc [C x E]; ro_b [E]; out_W [E x V];
 *   out_b [V].
 * With wtype = NMT_BF16 the values are rounded to bf16 (nearest, ties to
 * even) when copied; pass bf16-representable values to store them exactly. */
typedef struct {
  const float *emb_src, *enc_f_W, *enc_f_b, *enc_f_U, *enc_b_W, *enc_b_b, *enc_b_U;
  const float *att_Wc, *att_b, *init_W, *init_b;
  const float *emb_tgt, *g1_W, *g1_b, *g1_U, *att_Wq, *att_v;
  const float *g2_U, *g2_b, *g2_Wc, *ro_Ws, *ro_Wy, *ro_Wc, *ro_b, *out_W, *out_b;
} nmt_weights;

/* Copy the parameters to the current HIP device, re-laid-out for the
 * kernels.  With fp32 weights the model also holds two per-word tables, the
 * target embeddings times the first GRU's input weights [V x 3H] and times
 * the readout's word weights [V x E] (fp32, computed here: 1.4 GB at V =
 * 100k, H = 1024, E = 500), which the step reads in place of those
 * products.  The caller keeps ownership of the host arrays and may free them
 * on return.  Synchronous.  Errors: NMT_EINVAL (bad dims or null weight),
 * NMT_ENOMEM, NMT_EDEVICE. */
nmt_status nmt_model_create(const nmt_dims* dims, const nmt_weights* w, nmt_model** out);

/* Free the model (waits for the device first).  NULL is a no-op. */
void nmt_model_destroy(nmt_model* m);

/* Source initialisation (Section 5.1: the model is initialised with the
 * source sentence before any hypothesis is scored).  d_src_ids [S x Tpad]
 * int32 in [0, V_src) for positions below each length (padding positions
 * are ignored); h_len [S] host int32 in [1, Tpad].  Computes the
 * annotations, the attention keys and, if d_s0_out is not NULL, the initial
 * decoder states d_s0_out [S x H]; with fp32 weights also each position's
 * annotation times the second GRU's input weights and the readout's context
 * weights [S x Tpad x (3H + E), padded to a multiple of 128], which the step
 * mixes with the attention weights in place of those products of the
 * context.  The returned source owns its device
 * buffers; it may be used by nmt_score_batch on any stream once the work
 * enqueued here has completed in stream order.  Out-of-range source ids set
 * the model's device error flag (see nmt_stream_status) and read as id 0.
 * Errors: NMT_EINVAL, NMT_ENOMEM, NMT_EDEVICE. */
nmt_status nmt_encode(nmt_model* m, int32_t S, int32_t Tpad, const int32_t* d_src_ids,
                      const int32_t* h_len, float* d_s0_out, void* stream, nmt_source** out);

/* A source built from given annotations d_ctx [S x Tpad x 2H] (fp32; values
 * past each length are ignored) instead of the encoder: only the attention
 * keys (and, with fp32 weights, the annotations' projections) are computed.  For testing the decoder step in isolation. */
nmt_status nmt_source_from_annotations(nmt_model* m, int32_t S, int32_t Tpad, const float* d_ctx,
                                       const int32_t* h_len, void* stream, nmt_source** out);

/* Device views of a source: d_ctx [S x Tpad x 2H], d_pctx [S x Tpad x A]
 * (both zero past each length once the building work has completed).
 * Pointers stay valid until nmt_source_destroy.  Any output may be NULL. */
nmt_status nmt_source_info(const nmt_source* src, int32_t* S, int32_t* Tpad, const float** d_ctx,
                           const float** d_pctx);

/* Free a source (waits for the device first).  NULL is a no-op. */
void nmt_source_destroy(nmt_source* src);

/* Bytes of device workspace that serve nmt_score_batch (and
 * nmt_score_forest_step) for any batch of at most B rows: some smaller
 * batches need more than B itself (they split the vocabulary into more
 * slices), so this is the largest need over all sizes up to B.  0 for a NULL
 * model or B <= 0. */
size_t nmt_score_workspace_bytes(const nmt_model* m, int32_t B);

/* One batched decoder step: the forward step (H_i, P_i) <- NMT(H_{i-1}, E_i)
 * of Section 5.1 / Figure 2, for B rows.
 *   d_s_prev [B x H]  states H_{i-1} (fp32)
 *   d_y_prev [B]      previous target word of each row, -1 = sentence start
 *                     (the embedding lookups forming E_i)
 *   d_sent_id [B]     source sentence of each row, in [0, S)
 *   d_req [B]         requested next word of each row, in [0, V)
 *   d_logp [B]        out: log p(req | row), natural log, full vocabulary
 *   d_s_new [B x H]   out: new states H_i (may alias d_s_prev)
 *   d_logZ [B]        out, nullable: per-row log normaliser
 *   d_workspace       device scratch of at least
 *                     nmt_score_workspace_bytes(m, B) bytes, 256-byte aligned
 * Rows are independent: row b of every output depends only on row b of the
 * inputs.  B = 0 is a no-op.  The call allocates nothing.  Device-resident
 * ids out of range set the model's device error flag and give that row
 * logp = NaN (see nmt_stream_status).  Calls on different streams must use
 * different workspaces.  The source must come from nmt_encode or
 * nmt_source_from_annotations on this model (a source of a model with other
 * widths H or A, or that differs in whether it precomputes the context's
 * products, gives NMT_EINVAL).  Errors: NMT_EINVAL, NMT_EWORKSPACE,
 * NMT_EDEVICE. */
nmt_status nmt_score_batch(nmt_model* m, const nmt_source* src, int32_t B, const float* d_s_prev,
                           const int32_t* d_y_prev, const int32_t* d_sent_id, const int32_t* d_req,
                           float* d_logp, float* d_s_new, float* d_logZ, void* d_workspace,
                           size_t ws_bytes, void* stream);

/* nmt_score_batch that also writes the step's intermediates (each nullable):
 * d_alpha [B x Tpad] attention weights (zero past the length), d_c [B x 2H]
 * context, d_s1 [B x H] first-GRU state, d_t [B x E] readout. */
nmt_status nmt_score_batch_debug(nmt_model* m, const nmt_source* src, int32_t B,
                                 const float* d_s_prev, const int32_t* d_y_prev,
                                 const int32_t* d_sent_id, const int32_t* d_req, float* d_logp,
                                 float* d_s_new, float* d_logZ, void* d_workspace,
                                 size_t ws_bytes, void* stream, float* d_alpha, float* d_c,
                                 float* d_s1, float* d_t);

/* Size of the library's own scratch for nmt_score_batch_noalloc: 64 MiB per
 * device.  At the paper's dimensions (E = 500, H = A = 1024, V = 100k) that
 * holds the step of up to 2,304 rows with fp32 weights and 2,688 with bf16
 * weights. */
#define NMT_NOALLOC_SCRATCH_BYTES (64u << 20)

/* nmt_score_batch for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, results and errors as nmt_score_batch, without the
 * workspace: the step's scratch is a device array of
 * NMT_NOALLOC_SCRATCH_BYTES inside the library, one per device, set up by
 * nmt_model_create and held until the process ends.  The call allocates
 * nothing (no hipMalloc, hipFree or allocating library routine).
 * Every call on a device shares that device's array, whatever the model or
 * stream: calls that overlap in time on one device race and must be
 * serialised by the caller (one stream, or events).  The array keeps the
 * last call's contents; the step overwrites every byte it reads, so nothing
 * needs clearing.  Errors: those of nmt_score_batch, and NMT_EWORKSPACE
 * (nothing enqueued) when B rows need more than NMT_NOALLOC_SCRATCH_BYTES of
 * scratch; a B whose nmt_score_workspace_bytes is at most that always fits. */
nmt_status nmt_score_batch_noalloc(nmt_model* m, const nmt_source* src, int32_t B, const float* d_s_prev,
                                   const int32_t* d_y_prev, const int32_t* d_sent_id, const int32_t* d_req,
                                   float* d_logp, float* d_s_new, float* d_logZ, void* stream);

/* One level of the ScoreBatch procedure (Section 5.1, Figure 2): a batched
 * step whose rows take their input states from a device state pool by index
 * and may request several next words each.
 *   d_state_pool [pool_rows x H]  states; row b's input state is
 *                                 d_state_pool[d_state_row[b]] (so H_{i-1}
 *                                 is gathered on the device, never copied)
 *   d_state_row [B]               in [0, pool_rows)
 *   d_y_prev [B], d_sent_id [B]   as for nmt_score_batch
 *   d_req_off [B+1], d_req [nreq] requested words of row b are
 *                                 d_req[d_req_off[b] .. d_req_off[b+1])
 *                                 (CSR; offsets non-decreasing, in [0, nreq])
 *   d_logp [nreq]                 out: log p of each request under its row
 *   d_s_new [B x H]               out: new states (must not overlap the pool)
 *   d_logZ [B]                    out, nullable
 * Workspace as for nmt_score_batch with the same B.  Rows with an id out of
 * range or malformed offsets get NaN outputs and set the device error flag.
 * Errors: NMT_EINVAL, NMT_EWORKSPACE, NMT_EDEVICE. */
nmt_status nmt_score_forest_step(nmt_model* m, const nmt_source* src, int32_t B, const float* d_state_pool,
                                 int32_t pool_rows, const int32_t* d_state_row, const int32_t* d_y_prev,
                                 const int32_t* d_sent_id, const int32_t* d_req_off, const int32_t* d_req,
                                 int32_t nreq, float* d_logp, float* d_s_new, float* d_logZ, void* d_workspace,
                                 size_t ws_bytes, void* stream);

/* A forest of per-hypothesis prefix trees (Section 5.1, Figure 1), built on
 * the host from (hypothesis, target phrase) pairs.  Host-only; owns its
 * index arrays. */
typedef struct nmt_forest nmt_forest;

/* Build the forest.  Hypothesis h has last word h_hyp_word[h] (-1 = sentence
 * start) and source sentence h_hyp_sent[h]; pair p expands hypothesis
 * h_pair_hyp[p] by the words h_phrase_words[h_phrase_off[p] ..
 * h_phrase_off[p+1]) (h_phrase_off has n_pairs+1 entries starting at 0).
 * Phrases of one hypothesis that share a prefix share its tree nodes.
 * Level d (1-based) holds one step row per tree node of depth d-1 that has
 * children; the node's children are that row's requests, so the requests of
 * level d are the tree edges at depth d.  Errors: NMT_EINVAL, NMT_ERANGE
 * (a pair names a hypothesis outside [0, n_hyp)). */
nmt_status nmt_forest_build(int32_t n_hyp, const int32_t* h_hyp_word, const int32_t* h_hyp_sent, int32_t n_pairs,
                            const int32_t* h_pair_hyp, const int32_t* h_phrase_off, const int32_t* h_phrase_words,
                            nmt_forest** out);

/* Forest shape: depth (= longest phrase = number of steps), total rows and
 * requests over all levels, and the largest level's row count.  Any output
 * may be NULL. */
nmt_status nmt_forest_shape(const nmt_forest* f, int32_t* depth, int32_t* n_rows, int32_t* n_req, int32_t* max_rows);

/* Host copies of level d (1 <= d <= depth): row and request counts, and for
 * each row its input-state row (level 1: a hypothesis index; deeper levels:
 * the global row, counted over all levels, of the parent node's row), its
 * previous word, sentence and request offsets (rows+1), and the requested
 * words.  Any output may be NULL; arrays must hold the level's sizes. */
nmt_status nmt_forest_level(const nmt_forest* f, int32_t d, int32_t* rows, int32_t* nreq, int32_t* h_state_row,
                            int32_t* h_y_prev, int32_t* h_sent_id, int32_t* h_req_off, int32_t* h_req);

/* Host copy of each pair's path: [n_pairs x depth] global request index of
 * the pair's edge at every depth, -1 past the end of its phrase. */
nmt_status nmt_forest_pair_paths(const nmt_forest* f, int32_t* h_path);

/* Bytes of device workspace nmt_score_forest needs for forest f. */
size_t nmt_forest_workspace_bytes(const nmt_model* m, const nmt_forest* f);

/* The whole ScoreBatch procedure (Figure 2) on the device: one
 * nmt_score_forest_step per tree depth, each level's input states gathered
 * from the previous level's output rows, then each pair's log-probability
 * summed along its path.
 *   d_hyp_states [n_hyp x H]  the state that goes with each hypothesis' last
 *                             word (the same convention as d_s_prev)
 *   d_pair_logp [n_pairs]     out: log p(phrase | hypothesis)
 *   d_req_logp [n_req]        out, nullable: log p of every tree edge
 *   d_node_states [n_rows x H] out, nullable: the state each row produces
 *                             (for reuse as hypothesis states later)
 * Asynchronous on `stream`; f must stay alive until the work completes.
 * Errors: NMT_EINVAL, NMT_EWORKSPACE, NMT_EDEVICE. */
nmt_status nmt_score_forest(nmt_model* m, const nmt_source* src, const nmt_forest* f, const float* d_hyp_states,
                            float* d_pair_logp, float* d_req_logp, float* d_node_states, void* d_workspace,
                            size_t ws_bytes, void* stream);

/* Free a forest.  NULL is a no-op. */
void nmt_forest_destroy(nmt_forest* f);

/* ------------------------------------------------------- stack rescoring
 *
 * Section 5.3 (Figure 4): the decoder expands hypotheses with the NMT
 * feature set to 0; once a stack is complete, the direct predecessor of each
 * of its hypotheses -- (parent hypothesis, target phrase) -- is scored with
 * one ScoreBatch and the 0 is replaced by the model's log-probability.  A
 * rescorer keeps what that needs between stacks: for each of K models (the
 * models as separate features of Section 5), the decoder state that goes
 * with every hypothesis' last word, on the device, indexed by hypothesis id.
 * Hypotheses are numbered in creation order: 0..S-1 are the empty
 * hypotheses of the source's S sentences (state s0, sentence start), and
 * each nmt_rescore_stack call numbers its n hypotheses next. */
typedef struct nmt_rescorer nmt_rescorer;

/* models[k], srcs[k]: model k and its encoding of the S sentences (all
 * sources with the same S; all models with the same target vocabulary, on
 * the current device).  d_s0[k] [S x H_k]: model k's initial states (from
 * nmt_encode), copied.  capacity: most hypotheses the rescorer will hold,
 * S included; the state pools ([capacity x H_k] fp32 per model) are
 * allocated here.  The models and sources must outlive the rescorer.
 * Waits for `stream`.  Errors: NMT_EINVAL, NMT_ERANGE (K outside [1, 32],
 * capacity < S), NMT_ENOMEM, NMT_EDEVICE. */
nmt_status nmt_rescorer_create(int32_t K, nmt_model* const* models, const nmt_source* const* srcs,
                               const float* const* d_s0, int32_t capacity, void* stream, nmt_rescorer** out);

/* Rescore one stack of n hypotheses: hypothesis j expands existing
 * hypothesis h_parent[j] by the target words h_words[h_off[j] .. h_off[j+1])
 * (h_off[0] = 0; an empty phrase scores 0 and keeps the parent's state).
 * Identical (parent, phrase) predecessors are scored once; all of them go
 * through one prefix forest (nmt_score_forest) per model.
 *   h_logp [K x n]  out (host): h_logp[k*n + j] = log p(phrase_j | parent_j)
 *                   under model k (natural log, full vocabulary)
 *   h_ids [n]       out (host), nullable: the ids given to the n hypotheses
 * Each new hypothesis' states are stored for later stacks.  Runs on `stream`
 * and returns when the work is done (the decoder needs the scores); grows the
 * rescorer's own device scratch when a stack needs more.  Not thread-safe per
 * rescorer.  Errors: NMT_EINVAL, NMT_ERANGE (unknown parent, word outside the
 * vocabulary, pool full: nothing is scored then), NMT_ENOMEM, NMT_EDEVICE. */
nmt_status nmt_rescore_stack(nmt_rescorer* r, int32_t n, const int32_t* h_parent, const int32_t* h_off,
                             const int32_t* h_words, float* h_logp, int32_t* h_ids, void* stream);

/* Model k's state pool (device, [capacity x H_k], row = hypothesis id), the
 * number of hypotheses so far, and the shape of the last stack's forest
 * (unique predecessors, step rows, tree edges, depth).  Outputs nullable. */
nmt_status nmt_rescorer_info(const nmt_rescorer* r, int32_t k, const float** d_states, int32_t* n_hyp,
                             int32_t* last_pairs, int32_t* last_rows, int32_t* last_edges, int32_t* last_depth);

/* Free a rescorer and its state pools.  NULL is a no-op. */
void nmt_rescorer_destroy(nmt_rescorer* r);

/* ---------------------------------------------------------- several models
 *
 * Section 5: one or several models enter the phrase-based log-linear model
 * as separate instances of the same feature, each with its own tuned
 * weight, which makes several models behave like an ensemble (Section 6.2
 * uses two and three).  Section 6.3 replaces an ensemble by one model whose
 * parameters are the element-wise average of the members'. */

/* A new model whose every parameter is the weighted element-wise average
 * sum_k h_coef[k] * models[k] (h_coef NULL: 1/K each, as fp32); an fp32
 * model's per-word tables are computed anew from the averaged parameters.  The models
 * must have been created with identical nmt_dims on the current device.
 * Accumulation is fp32 in model order; results are stored in the models'
 * weight type (bf16 models keep every parameter, biases included, at a bf16
 * value, rounded to nearest even).  Runs on `stream` and waits for it; the
 * inputs stay untouched and owned by the caller; free the result with
 * nmt_model_destroy.  1 <= K <= 32.
 * Errors: NMT_EINVAL (NULL, mismatched models, non-finite coefficient),
 * NMT_ERANGE (K), NMT_ENOMEM, NMT_EDEVICE. */
nmt_status nmt_model_average(int32_t K, nmt_model* const* models, const float* h_coef, void* stream,
                             nmt_model** out);

/* Workspace bytes that serve nmt_score_ensemble for these K models and any
 * batch of at most B rows (the largest nmt_score_workspace_bytes over the
 * models; 0 for invalid arguments). */
size_t nmt_ensemble_workspace_bytes(int32_t K, nmt_model* const* models, int32_t B);

/* One batched step of the same B rows under K models (1 <= K <= 32), each
 * a separate feature: the models share the target vocabulary, the previous
 * words, the sentence ids and the requested words, and each has its own
 * encoded source and its own states.
 *   srcs[k]          model k's nmt_source (all with the same sentences)
 *   d_s_prev[k]      [B x H_k] model k's input states
 *   d_logp [K x B]   out: row k holds model k's log p of the requested word
 *   d_s_new[k]       [B x H_k] out: model k's new states (may alias d_s_prev[k])
 *   d_logZ [K x B]   out, nullable
 *   h_weights [K]    nullable (all 1): feature weights for d_score
 *   d_score [B]      out, nullable: sum_k h_weights[k] * d_logp[k][b], in
 *                    model order (the ensemble's share of the log-linear score)
 *   d_workspace      nmt_ensemble_workspace_bytes(K, models, B) bytes, 256-byte
 *                    aligned; the models run one after another on `stream` and
 *                    reuse it.
 * Row semantics, id checks and allocation behaviour are those of
 * nmt_score_batch for each model (check each model with nmt_stream_status).
 * Errors: NMT_EINVAL, NMT_ERANGE (K), NMT_EWORKSPACE, NMT_EDEVICE. */
nmt_status nmt_score_ensemble(int32_t K, nmt_model* const* models, const nmt_source* const* srcs, int32_t B,
                              const float* const* d_s_prev, const int32_t* d_y_prev, const int32_t* d_sent_id,
                              const int32_t* d_req, float* d_logp, float* const* d_s_new, float* d_logZ,
                              const float* h_weights, float* d_score, void* d_workspace, size_t ws_bytes,
                              void* stream);

/* Wait for `stream`, then report and clear the model's device error flag:
 * NMT_ERANGE if any call since the last check met an out-of-range id,
 * NMT_EDEVICE on a HIP error, else NMT_OK. */
nmt_status nmt_stream_status(nmt_model* m, void* stream);

/* Message for the last failed call on this thread ("" if none). */
const char* nmt_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* NMT_H */
