// forest_host.cpp -- the host side of the ScoreBatch procedure (Section 5.1,
// Figures 1 and 2): collapsing each hypothesis' target phrases into a
// prefix tree and laying the trees out as per-depth step rows, and the
// predecessor extraction of stack rescoring (Section 5.3, Figure 4).  Plain
// C++ with no device code, so it also builds alone (with the address and
// undefined-behaviour sanitizers in the tests).
//
// With the step's convention (input: previous word and the state before it;
// output: the distribution over the next word and the state after it), one
// step row serves a whole tree node: a node with children is a row whose
// input is the node's word (the hypothesis' last word for a root) and the
// state produced by its parent's row, and whose requested words are its
// children's words.  The requests of a level are the edges of the paper's
// per-depth dashed boxes; rows requesting the same parent state are not
// duplicated.
#include <stdint.h>

#include <string>
#include <unordered_map>
#include <vector>

#include "forest.hpp"

using namespace nmt;

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

}  // namespace

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

}  // extern "C"

namespace nmt {

void extract_predecessors(int32_t n, const int32_t* h_parent, const int32_t* h_off, const int32_t* h_words,
                          Predecessors* out) {
  std::unordered_map<std::string, int32_t> seen;
  out->pair_of.assign(n, 0);
  out->pair_hyp.clear();
  out->pair_off.assign(1, 0);
  out->pair_words.clear();
  for (int32_t j = 0; j < n; ++j) {
    const int32_t len = h_off[j + 1] - h_off[j];
    std::string key((const char*)&h_parent[j], 4);
    if (len > 0) key.append((const char*)(h_words + h_off[j]), (size_t)len * 4);
    auto it = seen.find(key);
    if (it != seen.end()) {
      out->pair_of[j] = it->second;
      continue;
    }
    const int32_t p = (int32_t)out->pair_hyp.size();
    seen.emplace(std::move(key), p);
    out->pair_of[j] = p;
    out->pair_hyp.push_back(h_parent[j]);
    if (len > 0) out->pair_words.insert(out->pair_words.end(), h_words + h_off[j], h_words + h_off[j + 1]);
    out->pair_off.push_back((int32_t)out->pair_words.size());
  }
}

void gather_plan(const nmt_forest* f, const Predecessors& P, int32_t n, int32_t first_id,
                 std::vector<int32_t>* plan) {
  plan->resize((size_t)2 * n);
  for (int32_t j = 0; j < n; ++j) {
    const int32_t p = P.pair_of[j], len = P.pair_off[p + 1] - P.pair_off[p];
    (*plan)[j] = len == 0 ? -(P.pair_hyp[p] + 1) : f->req_row[f->pair_path[(size_t)p * f->depth + len - 1]];
    (*plan)[n + j] = first_id + j;
  }
}

}  // namespace nmt
