// forest.hip -- the device side of the ScoreBatch procedure of the paper
// (Section 5.1, Figure 2) over a forest of per-hypothesis prefix trees
// (Figure 1), and of stack rescoring (Section 5.3, Figure 4).  The trees
// and their per-depth step rows are built on the host (forest_host.cpp);
// here every tree depth costs one batched decoder step, so the number of
// steps is the longest phrase length however many pairs there are.  Input
// states are gathered on the device from the previous level's output rows,
// so states stay in device memory across depths.
#include <stdint.h>

#include <vector>

#include "forest.hpp"
#include "internal.hpp"

using namespace nmt;

namespace {

__global__ void k_path_sum(int n_pairs, int depth, const int32_t* __restrict__ path, const float* __restrict__ logp,
                           float* __restrict__ out) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n_pairs) return;
  float s = 0.f;
  for (int k = 0; k < depth; ++k) {
    const int j = path[(int64_t)p * depth + k];
    if (j >= 0) s += logp[j];
  }
  out[p] = s;
}

struct ForestWs {
  size_t idx, logp, states, perm, tiles, ntiles, step, total;
  size_t n_idx;
};

size_t al256(size_t x) { return (x + 255) / 256 * 256; }

}  // namespace

// Implemented in api.hip.
nmt_status nmt_internal_score_step(nmt_model* m, const nmt_source* src, int32_t B, const float* pool,
                                   int32_t pool_rows, const int32_t* state_row, const int32_t* y_prev,
                                   const int32_t* sent_id, const int32_t* req_off, const int32_t* req, int32_t nreq,
                                   float* logp, float* s_new, void* ws, size_t ws_bytes, hipStream_t st,
                                   const AttnGroups* grp);
bool nmt_internal_group_levels(const nmt_model* m, const nmt_source* src, GroupLevel* lv, int n, hipStream_t st,
                               hipError_t* err);
int32_t nmt_internal_hidden(const nmt_model* m);
int32_t nmt_internal_sentences(const nmt_source* src);
int32_t nmt_internal_vocab(const nmt_model* m);
int nmt_internal_device(const nmt_model* m);

static ForestWs forest_ws(const nmt_model* m, const nmt_forest* f) {
  ForestWs L{};
  // index arrays: state_row, y_prev, sent (n_rows each), req_off (n_rows + depth), req (n_req), pair_path
  L.n_idx = (size_t)3 * f->n_rows + (f->n_rows + f->depth) + f->n_req + (size_t)f->n_pairs * f->depth;
  size_t off = 0;
  L.idx = off;
  off += al256(L.n_idx * 4);
  L.logp = off;
  off += al256((size_t)f->n_req * 4);
  L.states = off;
  off += al256((size_t)f->n_rows * nmt_internal_hidden(m) * 4);
  // every level's grouping of rows by sentence (at most one tile per row)
  L.perm = off;
  off += al256((size_t)f->n_rows * 4);
  L.tiles = off;
  off += al256((size_t)f->n_rows * 16);
  L.ntiles = off;
  off += al256((size_t)f->depth * 4);
  L.step = off;
  off += al256(nmt_score_workspace_bytes(m, f->max_rows));
  L.total = off;
  return L;
}

extern "C" {

size_t nmt_forest_workspace_bytes(const nmt_model* m, const nmt_forest* f) {
  if (!m || !f) return 0;
  return forest_ws(m, f).total;
}

nmt_status nmt_score_forest(nmt_model* m, const nmt_source* src, const nmt_forest* f, const float* d_hyp_states,
                            float* d_pair_logp, float* d_req_logp, float* d_node_states, void* d_workspace,
                            size_t ws_bytes, void* stream) {
  if (!m || !src || !f) return forest_fail(NMT_EINVAL, "NULL model, source or forest");
  if (f->n_pairs == 0) return NMT_OK;
  if (!d_pair_logp || (f->n_hyp > 0 && !d_hyp_states)) return forest_fail(NMT_EINVAL, "a required pointer is NULL");
  if (((uintptr_t)d_hyp_states & 15) || ((uintptr_t)d_node_states & 15))
    return forest_fail(NMT_EINVAL, "state arrays must be 16-byte aligned");
  if (!d_workspace || ((uintptr_t)d_workspace & 255))
    return forest_fail(NMT_EINVAL, "workspace must be 256-byte aligned");
  const ForestWs L = forest_ws(m, f);
  if (ws_bytes < L.total) return forest_fail(NMT_EWORKSPACE, "workspace too small for this forest");
  hipStream_t st = (hipStream_t)stream;
  const int H = nmt_internal_hidden(m);
  char* ws = (char*)d_workspace;
  int32_t* idx = (int32_t*)(ws + L.idx);
  float* logp = d_req_logp ? d_req_logp : (float*)(ws + L.logp);
  float* states = d_node_states ? d_node_states : (float*)(ws + L.states);
  // one upload of every level's index arrays (from the forest, which the
  // caller keeps alive until this work has completed)
  int32_t* d_state_row = idx;
  int32_t* d_y = d_state_row + f->n_rows;
  int32_t* d_sent = d_y + f->n_rows;
  int32_t* d_off = d_sent + f->n_rows;
  int32_t* d_req = d_off + f->n_rows + f->depth;
  int32_t* d_path = d_req + f->n_req;
  hipError_t e = hipMemcpyAsync(idx, f->upload.data(), f->upload.size() * 4, hipMemcpyHostToDevice, st);
  if (e != hipSuccess) return forest_fail(NMT_EDEVICE, hipGetErrorString(e));
  // the attention's grouping of rows by sentence, for all levels at once;
  // when every row is of one (valid) sentence, as in the stack rescoring of
  // one sentence, no grouping: each level's attention tiles its rows in order
  int32_t s_one = f->n_rows > 0 ? f->sent[0] : -1;
  for (int32_t i = 1; i < f->n_rows && s_one >= 0; ++i)
    if (f->sent[i] != s_one) s_one = -1;
  if (s_one < 0 || s_one >= nmt_internal_sentences(src)) s_one = -1;
  std::vector<GroupLevel> lv((size_t)f->depth);
  for (int d = 1; d <= f->depth; ++d) {
    const int32_t r0 = f->row_base[d - 1];
    lv[d - 1] = GroupLevel{f->rows_lv[d - 1], 0, d_sent + r0,
                           AttnGroups{(int32_t*)(ws + L.perm) + r0, (int4*)(ws + L.tiles) + r0,
                                      (int32_t*)(ws + L.ntiles) + (d - 1), s_one}};
  }
  const bool grouped = s_one >= 0 || nmt_internal_group_levels(m, src, lv.data(), f->depth, st, &e);
  if (e != hipSuccess) return forest_fail(NMT_EDEVICE, hipGetErrorString(e));
  for (int d = 1; d <= f->depth; ++d) {
    const int32_t r0 = f->row_base[d - 1], q0 = f->req_base[d - 1];
    const float* pool = d == 1 ? d_hyp_states : states;
    const int32_t pool_rows = d == 1 ? f->n_hyp : f->n_rows;
    nmt_status rc = nmt_internal_score_step(m, src, f->rows_lv[d - 1], pool, pool_rows, d_state_row + r0, d_y + r0,
                                            d_sent + r0, d_off + f->off_base[d - 1], d_req + q0, f->req_lv[d - 1],
                                            logp + q0, states + (int64_t)r0 * H, ws + L.step, ws_bytes - L.step, st,
                                            grouped ? &lv[d - 1].grp : nullptr);
    if (rc != NMT_OK) return rc;
  }
  hipLaunchKernelGGL(k_path_sum, dim3(ceil_div(f->n_pairs, 256)), dim3(256), 0, st, f->n_pairs, f->depth, d_path,
                     logp, d_pair_logp);
  e = hipGetLastError();
  if (e != hipSuccess) return forest_fail(NMT_EDEVICE, hipGetErrorString(e));
  return NMT_OK;
}

}  // extern "C"

// ------------------------------------------------------- stack rescoring
//
// Section 5.3 (Figure 4): hypotheses are expanded without the NMT feature,
// and when a stack is complete the direct predecessor of each of its
// hypotheses -- (parent hypothesis, target phrase) -- is scored with one
// ScoreBatch over all of them; identical predecessors are scored once.  The
// rescorer keeps, per model, the decoder state that goes with every
// hypothesis' last word in a device pool indexed by hypothesis id, so a
// stack's forest reads its roots' states straight from the pool and the new
// hypotheses' states are gathered into it from the forest's output rows.

namespace {

// dst[dst_row[j]] = src_row[j] >= 0 ? nodes[src_row[j]] : pool[-src_row[j] - 1], one block per row.
__global__ void k_gather_states(int n, int H, const int32_t* __restrict__ src_row, const int32_t* __restrict__ dst_row,
                                const float* __restrict__ nodes, float* __restrict__ pool) {
  const int j = blockIdx.x;
  if (j >= n) return;
  const int32_t s = src_row[j];
  const float* from = s >= 0 ? nodes + (int64_t)s * H : pool + (int64_t)(-s - 1) * H;
  float* to = pool + (int64_t)dst_row[j] * H;
  for (int k = threadIdx.x * 4; k < H; k += blockDim.x * 4) *(float4*)(to + k) = *(const float4*)(from + k);
}

struct DevBuf {
  void* p = nullptr;
  size_t cap = 0;
  // Grows to at least `bytes` (contents are not kept); the stream is idle here.
  hipError_t ensure(size_t bytes) {
    if (bytes <= cap) return hipSuccess;
    device_free(p);
    p = nullptr;
    cap = 0;
    const size_t want = bytes + bytes / 4 + 4096;
    hipError_t e = device_malloc(&p, want);
    if (e == hipSuccess) cap = want;
    return e;
  }
  void release() {
    device_free(p);
    p = nullptr;
    cap = 0;
  }
};

}  // namespace

struct nmt_rescorer {
  int32_t K = 0, S = 0, capacity = 0, n_hyp = 0;
  std::vector<nmt_model*> models;
  std::vector<const nmt_source*> srcs;
  std::vector<int32_t> H;
  std::vector<float*> pool;            // per model [capacity x H_k], owned
  std::vector<int32_t> last_word, sent;  // per hypothesis (host)
  DevBuf ws, nodes, pair_logp, gather;
  std::vector<float> h_pair_logp;
  std::vector<int32_t> h_gather;
  int32_t last_pairs = 0, last_rows = 0, last_depth = 0, last_edges = 0;
};

extern "C" {

nmt_status nmt_rescorer_create(int32_t K, nmt_model* const* models, const nmt_source* const* srcs,
                               const float* const* d_s0, int32_t capacity, void* stream, nmt_rescorer** out) {
  if (!out) return forest_fail(NMT_EINVAL, "NULL output");
  *out = nullptr;
  if (K < 1 || K > 32) return forest_fail(NMT_ERANGE, "K must be in [1, 32]");
  if (!models || !srcs || !d_s0) return forest_fail(NMT_EINVAL, "NULL argument");
  int32_t S = 0;
  for (int k = 0; k < K; ++k) {
    if (!models[k] || !srcs[k] || !d_s0[k]) return forest_fail(NMT_EINVAL, "a model, source or s0 is NULL");
    if (((uintptr_t)d_s0[k] & 15)) return forest_fail(NMT_EINVAL, "s0 arrays must be 16-byte aligned");
    int32_t Sk = 0;
    nmt_source_info(srcs[k], &Sk, nullptr, nullptr, nullptr);
    if (k == 0) S = Sk;
    if (Sk != S) return forest_fail(NMT_EINVAL, "sources hold different numbers of sentences");
    if (nmt_internal_vocab(models[k]) != nmt_internal_vocab(models[0]) ||
        nmt_internal_device(models[k]) != nmt_internal_device(models[0]))
      return forest_fail(NMT_EINVAL, "models differ in target vocabulary or device");
  }
  if (capacity < S) return forest_fail(NMT_ERANGE, "capacity must hold at least the S empty hypotheses");
  hipStream_t st = (hipStream_t)stream;
  nmt_rescorer* r = new nmt_rescorer();
  r->K = K;
  r->S = S;
  r->capacity = capacity;
  r->n_hyp = S;
  r->models.assign(models, models + K);
  r->srcs.assign(srcs, srcs + K);
  hipError_t e = hipSuccess;
  for (int k = 0; k < K && e == hipSuccess; ++k) {
    const int32_t H = nmt_internal_hidden(models[k]);
    r->H.push_back(H);
    float* p = nullptr;
    e = device_malloc((void**)&p, (size_t)capacity * H * 4);
    if (e == hipSuccess) {
      r->pool.push_back(p);
      // hypotheses 0..S-1: the empty hypothesis of each sentence, state s0
      e = hipMemcpyAsync(p, d_s0[k], (size_t)S * H * 4, hipMemcpyDeviceToDevice, st);
    }
  }
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) {
    nmt_rescorer_destroy(r);
    return forest_fail(e == hipErrorOutOfMemory ? NMT_ENOMEM : NMT_EDEVICE, hipGetErrorString(e));
  }
  r->last_word.assign(S, -1);  // sentence start
  r->sent.resize(S);
  for (int32_t s = 0; s < S; ++s) r->sent[s] = s;
  *out = r;
  return NMT_OK;
}

void nmt_rescorer_destroy(nmt_rescorer* r) {
  if (!r) return;
  (void)hipDeviceSynchronize();
  for (float* p : r->pool) device_free(p);
  r->ws.release();
  r->nodes.release();
  r->pair_logp.release();
  r->gather.release();
  delete r;
}

nmt_status nmt_rescore_stack(nmt_rescorer* r, int32_t n, const int32_t* h_parent, const int32_t* h_off,
                             const int32_t* h_words, float* h_logp, int32_t* h_ids, void* stream) {
  if (!r) return forest_fail(NMT_EINVAL, "NULL rescorer");
  if (n < 0) return forest_fail(NMT_EINVAL, "negative stack size");
  if (n == 0) return NMT_OK;
  if (!h_parent || !h_off || !h_logp) return forest_fail(NMT_EINVAL, "a required host array is NULL");
  if (h_off[0] != 0) return forest_fail(NMT_EINVAL, "phrase offsets must start at 0");
  if (n > r->capacity - r->n_hyp) return forest_fail(NMT_ERANGE, "the state pool is full");
  const int32_t V = nmt_internal_vocab(r->models[0]);
  for (int32_t j = 0; j < n; ++j) {
    if (h_parent[j] < 0 || h_parent[j] >= r->n_hyp) return forest_fail(NMT_ERANGE, "parent is not an existing hypothesis");
    if (h_off[j + 1] < h_off[j]) return forest_fail(NMT_EINVAL, "phrase offsets must not decrease");
  }
  if (h_off[n] > 0 && !h_words) return forest_fail(NMT_EINVAL, "phrase words are NULL");
  for (int32_t i = 0; i < h_off[n]; ++i)
    if (h_words[i] < 0 || h_words[i] >= V) return forest_fail(NMT_ERANGE, "phrase word out of the vocabulary");
  hipStream_t st = (hipStream_t)stream;

  // Predecessor extraction: identical (parent, phrase) pairs are one entry of L.
  Predecessors P;
  extract_predecessors(n, h_parent, h_off, h_words, &P);
  const int32_t np = (int32_t)P.pair_hyp.size();
  // ScoreBatch over all predecessors: hypothesis ids index the forest's roots and the pools.
  nmt_forest* f = nullptr;
  nmt_status rc = nmt_forest_build(r->n_hyp, r->last_word.data(), r->sent.data(), np, P.pair_hyp.data(),
                                   P.pair_off.data(), P.pair_words.data(), &f);
  if (rc != NMT_OK) return rc;
  const int32_t depth = f->depth, n_rows = f->n_rows;
  int32_t maxH = 0;
  size_t ws_need = 0;
  for (int k = 0; k < r->K; ++k) {
    maxH = r->H[k] > maxH ? r->H[k] : maxH;
    const size_t b = nmt_forest_workspace_bytes(r->models[k], f);
    ws_need = b > ws_need ? b : ws_need;
  }
  // A buffer that grows is freed first: wait for the stream only then (the
  // previous call's work ended with a synchronisation of its own).
  const size_t nodes_need = (size_t)n_rows * maxH * 4, logp_need = (size_t)r->K * np * 4,
               gather_need = (size_t)2 * n * 4;
  const bool grow = ws_need > r->ws.cap || nodes_need > r->nodes.cap || logp_need > r->pair_logp.cap ||
                    gather_need > r->gather.cap;
  hipError_t e = grow ? hipStreamSynchronize(st) : hipSuccess;
  if (e == hipSuccess) e = r->ws.ensure(ws_need);
  if (e == hipSuccess) e = r->nodes.ensure(nodes_need);
  if (e == hipSuccess) e = r->pair_logp.ensure(logp_need);
  if (e == hipSuccess) e = r->gather.ensure(gather_need);
  if (e != hipSuccess) {
    nmt_forest_destroy(f);
    return forest_fail(e == hipErrorOutOfMemory ? NMT_ENOMEM : NMT_EDEVICE, hipGetErrorString(e));
  }
  // Where each new hypothesis' state comes from, and where it goes.
  gather_plan(f, P, n, r->n_hyp, &r->h_gather);
  int32_t* d_gather = (int32_t*)r->gather.p;
  float* d_pair_logp = (float*)r->pair_logp.p;
  e = hipMemcpyAsync(d_gather, r->h_gather.data(), (size_t)2 * n * 4, hipMemcpyHostToDevice, st);
  for (int k = 0; k < r->K && e == hipSuccess && rc == NMT_OK; ++k) {
    rc = nmt_score_forest(r->models[k], r->srcs[k], f, r->pool[k], d_pair_logp + (size_t)k * np, nullptr,
                          (float*)r->nodes.p, r->ws.p, r->ws.cap, stream);
    if (rc != NMT_OK) break;
    hipLaunchKernelGGL(k_gather_states, dim3(n), dim3(256), 0, st, n, r->H[k], d_gather, d_gather + n,
                       (const float*)r->nodes.p, r->pool[k]);
    e = hipGetLastError();
  }
  r->h_pair_logp.resize((size_t)r->K * np);
  if (e == hipSuccess && rc == NMT_OK)
    e = hipMemcpyAsync(r->h_pair_logp.data(), d_pair_logp, (size_t)r->K * np * 4, hipMemcpyDeviceToHost, st);
  const hipError_t es = hipStreamSynchronize(st);
  if (e == hipSuccess) e = es;
  r->last_pairs = np;
  r->last_rows = n_rows;
  r->last_depth = depth;
  r->last_edges = f->n_req;
  nmt_forest_destroy(f);
  if (rc != NMT_OK) return rc;
  if (e != hipSuccess) return forest_fail(NMT_EDEVICE, hipGetErrorString(e));
  // Look up p for each hypothesis' predecessor; number the new hypotheses.
  for (int k = 0; k < r->K; ++k)
    for (int32_t j = 0; j < n; ++j) h_logp[(size_t)k * n + j] = r->h_pair_logp[(size_t)k * np + P.pair_of[j]];
  for (int32_t j = 0; j < n; ++j) {
    const int32_t len = h_off[j + 1] - h_off[j];
    r->last_word.push_back(len > 0 ? h_words[h_off[j + 1] - 1] : r->last_word[h_parent[j]]);
    r->sent.push_back(r->sent[h_parent[j]]);
    if (h_ids) h_ids[j] = r->n_hyp + j;
  }
  r->n_hyp += n;
  return NMT_OK;
}

nmt_status nmt_rescorer_info(const nmt_rescorer* r, int32_t k, const float** d_states, int32_t* n_hyp,
                             int32_t* last_pairs, int32_t* last_rows, int32_t* last_edges, int32_t* last_depth) {
  if (!r) return forest_fail(NMT_EINVAL, "NULL rescorer");
  if (k < 0 || k >= r->K) return forest_fail(NMT_ERANGE, "model index out of range");
  if (d_states) *d_states = r->pool[k];
  if (n_hyp) *n_hyp = r->n_hyp;
  if (last_pairs) *last_pairs = r->last_pairs;
  if (last_rows) *last_rows = r->last_rows;
  if (last_edges) *last_edges = r->last_edges;
  if (last_depth) *last_depth = r->last_depth;
  return NMT_OK;
}

}  // extern "C"
