// forest.hip -- the ScoreBatch procedure of the paper (Section 5.1,
// Figure 2) over a forest of per-hypothesis prefix trees (Figure 1).
//
// Given (hypothesis, target phrase) pairs, the phrases of each hypothesis
// are collapsed into a prefix tree, and every tree depth costs one batched
// decoder step, so the number of steps is the longest phrase length however
// many pairs there are.  With the step's convention (input: previous word and
// the state before it; output: the distribution over the next word and the
// state after it), one step row serves a whole tree node: a node with
// children is a row whose input is the node's word (the hypothesis' last word
// for a root) and the state produced by its parent's row, and whose requested
// words are its children's words.  The requests of a level are the edges of
// the paper's per-depth dashed boxes; rows requesting the same parent state
// are not duplicated.  Input states are gathered on the device from the
// previous level's output rows, so states stay in device memory across
// depths.
#include <stdint.h>

#include <string>
#include <unordered_map>
#include <vector>

#include "../../include/nmt.h"
#include "internal.hpp"

using namespace nmt;

struct nmt_forest {
  int32_t n_hyp = 0, n_pairs = 0, depth = 0;
  int32_t n_rows = 0, n_req = 0, max_rows = 0;
  std::vector<int32_t> rows_lv, req_lv;      // per level (1-based level d at index d-1)
  std::vector<int32_t> row_base, req_base;   // first global row / request of each level
  std::vector<int32_t> off_base;             // first offset entry of each level
  // per global row
  std::vector<int32_t> state_row;  // level 1: hypothesis index; deeper: global row of the parent node's row
  std::vector<int32_t> y_prev, sent;
  std::vector<int32_t> req_off;   // per level, rows+1 offsets local to the level
  std::vector<int32_t> req;       // per global request: the requested word
  std::vector<int32_t> req_row;   // per global request: its global row
  std::vector<int32_t> pair_path; // [n_pairs x depth] global request index per depth, -1 past the end
  std::vector<int32_t> upload;    // all of the above index arrays, in the device workspace order
};

namespace nmt {
nmt_status forest_fail(nmt_status st, const char* msg);
}

namespace {

struct Node {
  int32_t parent;  // -1 for roots
  int32_t word;    // edge word (roots: the hypothesis' last word)
  int32_t hyp;
  int32_t depth;
  int32_t row = -1;               // global row of this node's step (if it has children)
  std::vector<int32_t> children;  // in creation order
  std::vector<int32_t> child_req; // global request index of each child edge
};

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
  size_t idx, logp, states, step, total;
  size_t n_idx;
};

size_t al256(size_t x) { return (x + 255) / 256 * 256; }

}  // namespace

// Implemented in api.hip.
nmt_status nmt_internal_score_step(nmt_model* m, const nmt_source* src, int32_t B, const float* pool,
                                   int32_t pool_rows, const int32_t* state_row, const int32_t* y_prev,
                                   const int32_t* sent_id, const int32_t* req_off, const int32_t* req, int32_t nreq,
                                   float* logp, float* s_new, void* ws, size_t ws_bytes, hipStream_t st);
int32_t nmt_internal_hidden(const nmt_model* m);

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
  L.step = off;
  off += al256(nmt_score_workspace_bytes(m, f->max_rows));
  L.total = off;
  return L;
}

extern "C" {

nmt_status nmt_forest_build(int32_t n_hyp, const int32_t* h_hyp_word, const int32_t* h_hyp_sent, int32_t n_pairs,
                            const int32_t* h_pair_hyp, const int32_t* h_phrase_off, const int32_t* h_phrase_words,
                            nmt_forest** out) {
  if (!out) return forest_fail(NMT_EINVAL, "NULL output");
  *out = nullptr;
  if (n_hyp < 0 || n_pairs < 0) return forest_fail(NMT_EINVAL, "negative count");
  if ((n_hyp > 0 && (!h_hyp_word || !h_hyp_sent)) || (n_pairs > 0 && (!h_pair_hyp || !h_phrase_off)))
    return forest_fail(NMT_EINVAL, "a required host array is NULL");
  if (n_pairs > 0 && h_phrase_off[0] != 0) return forest_fail(NMT_EINVAL, "phrase offsets must start at 0");
  for (int p = 0; p < n_pairs; ++p) {
    if (h_pair_hyp[p] < 0 || h_pair_hyp[p] >= n_hyp) return forest_fail(NMT_ERANGE, "pair hypothesis out of range");
    if (h_phrase_off[p + 1] < h_phrase_off[p]) return forest_fail(NMT_EINVAL, "phrase offsets must not decrease");
  }
  if (n_pairs > 0 && h_phrase_off[n_pairs] > 0 && !h_phrase_words)
    return forest_fail(NMT_EINVAL, "phrase words are NULL");

  nmt_forest* f = new nmt_forest();
  f->n_hyp = n_hyp;
  f->n_pairs = n_pairs;
  // prefix trees: one root per hypothesis with a non-empty phrase
  std::vector<Node> nodes;
  std::vector<int32_t> root(n_hyp, -1);
  std::unordered_map<uint64_t, int32_t> child_of;  // (node, word) -> child node
  std::vector<std::vector<int32_t>> pair_nodes(n_pairs);
  int32_t depth = 0;
  for (int p = 0; p < n_pairs; ++p) {
    const int h = h_pair_hyp[p], len = h_phrase_off[p + 1] - h_phrase_off[p];
    if (len == 0) continue;
    if (root[h] < 0) {
      root[h] = (int32_t)nodes.size();
      nodes.push_back(Node{-1, h_hyp_word[h], h, 0});
    }
    int32_t cur = root[h];
    for (int k = 0; k < len; ++k) {
      const int32_t w = h_phrase_words[h_phrase_off[p] + k];
      const uint64_t key = ((uint64_t)(uint32_t)cur << 32) | (uint32_t)w;
      auto it = child_of.find(key);
      int32_t nxt;
      if (it == child_of.end()) {
        nxt = (int32_t)nodes.size();
        nodes.push_back(Node{cur, w, h, nodes[cur].depth + 1});
        nodes[cur].children.push_back(nxt);
        child_of.emplace(key, nxt);
      } else {
        nxt = it->second;
      }
      pair_nodes[p].push_back(nxt);
      cur = nxt;
    }
    if (len > depth) depth = len;
  }
  f->depth = depth;
  // levels: level d holds the nodes of depth d-1 that have children, in creation order
  std::vector<std::vector<int32_t>> by_depth(depth + 1);
  for (int32_t i = 0; i < (int32_t)nodes.size(); ++i)
    if (nodes[i].depth < depth && !nodes[i].children.empty()) by_depth[nodes[i].depth].push_back(i);
  f->rows_lv.resize(depth);
  f->req_lv.resize(depth);
  f->row_base.resize(depth);
  f->req_base.resize(depth);
  f->off_base.resize(depth);
  int32_t grow = 0, greq = 0, goff = 0;
  for (int d = 1; d <= depth; ++d) {
    const auto& lv = by_depth[d - 1];
    f->row_base[d - 1] = grow;
    f->req_base[d - 1] = greq;
    f->off_base[d - 1] = goff;
    f->rows_lv[d - 1] = (int32_t)lv.size();
    int32_t local = 0;
    for (int32_t id : lv) {
      Node& n = nodes[id];
      n.row = grow++;
      f->state_row.push_back(n.parent < 0 ? n.hyp : nodes[n.parent].row);
      f->y_prev.push_back(n.word);
      f->sent.push_back(h_hyp_sent[n.hyp]);
      f->req_off.push_back(local);
      for (int32_t c : n.children) {
        n.child_req.push_back(greq++);
        f->req.push_back(nodes[c].word);
        f->req_row.push_back(n.row);
        ++local;
      }
    }
    f->req_off.push_back(local);
    goff += (int32_t)lv.size() + 1;
    f->req_lv[d - 1] = local;
    if ((int32_t)lv.size() > f->max_rows) f->max_rows = (int32_t)lv.size();
  }
  f->n_rows = grow;
  f->n_req = greq;
  // each pair's path: the request of its edge at every depth
  f->pair_path.assign((size_t)n_pairs * depth, -1);
  for (int p = 0; p < n_pairs; ++p)
    for (size_t k = 0; k < pair_nodes[p].size(); ++k) {
      const Node& child = nodes[pair_nodes[p][k]];
      const Node& par = nodes[child.parent];
      for (size_t c = 0; c < par.children.size(); ++c)
        if (par.children[c] == pair_nodes[p][k]) f->pair_path[(size_t)p * depth + k] = par.child_req[c];
    }
  for (const std::vector<int32_t>* v : {&f->state_row, &f->y_prev, &f->sent, &f->req_off, &f->req, &f->pair_path})
    f->upload.insert(f->upload.end(), v->begin(), v->end());
  *out = f;
  return NMT_OK;
}

void nmt_forest_destroy(nmt_forest* f) { delete f; }

nmt_status nmt_forest_shape(const nmt_forest* f, int32_t* depth, int32_t* n_rows, int32_t* n_req, int32_t* max_rows) {
  if (!f) return forest_fail(NMT_EINVAL, "NULL forest");
  if (depth) *depth = f->depth;
  if (n_rows) *n_rows = f->n_rows;
  if (n_req) *n_req = f->n_req;
  if (max_rows) *max_rows = f->max_rows;
  return NMT_OK;
}

nmt_status nmt_forest_level(const nmt_forest* f, int32_t d, int32_t* rows, int32_t* nreq, int32_t* h_state_row,
                            int32_t* h_y_prev, int32_t* h_sent_id, int32_t* h_req_off, int32_t* h_req) {
  if (!f) return forest_fail(NMT_EINVAL, "NULL forest");
  if (d < 1 || d > f->depth) return forest_fail(NMT_EINVAL, "level out of range");
  const int32_t R = f->rows_lv[d - 1], Q = f->req_lv[d - 1], r0 = f->row_base[d - 1], q0 = f->req_base[d - 1];
  if (rows) *rows = R;
  if (nreq) *nreq = Q;
  for (int32_t i = 0; i < R; ++i) {
    if (h_state_row) h_state_row[i] = f->state_row[r0 + i];
    if (h_y_prev) h_y_prev[i] = f->y_prev[r0 + i];
    if (h_sent_id) h_sent_id[i] = f->sent[r0 + i];
  }
  if (h_req_off)
    for (int32_t i = 0; i <= R; ++i) h_req_off[i] = f->req_off[f->off_base[d - 1] + i];
  if (h_req)
    for (int32_t j = 0; j < Q; ++j) h_req[j] = f->req[q0 + j];
  return NMT_OK;
}

nmt_status nmt_forest_pair_paths(const nmt_forest* f, int32_t* h_path) {
  if (!f || !h_path) return forest_fail(NMT_EINVAL, "NULL argument");
  for (size_t i = 0; i < f->pair_path.size(); ++i) h_path[i] = f->pair_path[i];
  return NMT_OK;
}

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
  for (int d = 1; d <= f->depth; ++d) {
    const int32_t r0 = f->row_base[d - 1], q0 = f->req_base[d - 1];
    const float* pool = d == 1 ? d_hyp_states : states;
    const int32_t pool_rows = d == 1 ? f->n_hyp : f->n_rows;
    nmt_status rc = nmt_internal_score_step(m, src, f->rows_lv[d - 1], pool, pool_rows, d_state_row + r0, d_y + r0,
                                            d_sent + r0, d_off + f->off_base[d - 1], d_req + q0, f->req_lv[d - 1],
                                            logp + q0, states + (int64_t)r0 * H, ws + L.step, ws_bytes - L.step, st);
    if (rc != NMT_OK) return rc;
  }
  hipLaunchKernelGGL(k_path_sum, dim3(ceil_div(f->n_pairs, 256)), dim3(256), 0, st, f->n_pairs, f->depth, d_path,
                     logp, d_pair_logp);
  e = hipGetLastError();
  if (e != hipSuccess) return forest_fail(NMT_EDEVICE, hipGetErrorString(e));
  return NMT_OK;
}

}  // extern "C"
