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

#include <vector>

#include "forest.hpp"

using namespace nmt;

namespace {

// Open-addressing table from 64-bit keys to int32 values (linear probing,
// load factor at most 1/2).  All of one build's entries live in two flat
// arrays, so a stack of thousands of phrases costs no per-node allocation.
class FlatMap {
 public:
  static constexpr uint64_t kEmpty = ~0ull;
  void reset(size_t n) {
    size_t cap = 16;
    while (cap < 2 * n) cap <<= 1;
    key_.assign(cap, kEmpty);
    val_.resize(cap);
    mask_ = cap - 1;
  }
  // The value slot of key k (k != kEmpty); *fresh tells whether it was just added.
  int32_t& slot(uint64_t k, bool* fresh) {
    size_t i = mix(k) & mask_;
    while (key_[i] != kEmpty && key_[i] != k) i = (i + 1) & mask_;
    *fresh = key_[i] == kEmpty;
    key_[i] = k;
    return val_[i];
  }
  static uint64_t mix(uint64_t x) {  // the splitmix64 finaliser
    x ^= x >> 30;
    x *= 0xbf58476d1ce4e5b9ull;
    x ^= x >> 27;
    x *= 0x94d049bb133111ebull;
    return x ^ (x >> 31);
  }

 private:
  std::vector<uint64_t> key_;
  std::vector<int32_t> val_;
  size_t mask_ = 0;
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
  const int32_t n_words = n_pairs > 0 ? h_phrase_off[n_pairs] : 0;
  // Prefix trees: one root per hypothesis with a non-empty phrase.  Nodes are
  // numbered in creation order; a node's children form a list in creation
  // order (first_child / next_sibling, last_child for appending).
  std::vector<int32_t> parent, word, hyp, ndepth, first_child, last_child, next_sibling;
  const size_t cap = (size_t)n_pairs + n_words;
  for (auto* v : {&parent, &word, &hyp, &ndepth, &first_child, &last_child, &next_sibling}) v->reserve(cap);
  auto add_node = [&](int32_t par, int32_t w, int32_t h, int32_t d) {
    const int32_t id = (int32_t)parent.size();
    parent.push_back(par);
    word.push_back(w);
    hyp.push_back(h);
    ndepth.push_back(d);
    first_child.push_back(-1);
    last_child.push_back(-1);
    next_sibling.push_back(-1);
    if (par >= 0) {
      if (last_child[par] < 0) first_child[par] = id;
      else next_sibling[last_child[par]] = id;
      last_child[par] = id;
    }
    return id;
  };
  // Keys: (node << 32 | word) for an edge, (1 << 63 | hypothesis << 32) for a
  // root; node ids stay below 2^31, so the two kinds never collide.
  FlatMap edges;
  edges.reset(cap);
  std::vector<int32_t> pair_node((size_t)n_words);  // node reached by each phrase word
  int32_t depth = 0;
  for (int p = 0; p < n_pairs; ++p) {
    const int32_t h = h_pair_hyp[p], o = h_phrase_off[p], len = h_phrase_off[p + 1] - o;
    if (len == 0) continue;
    bool fresh = false;
    int32_t& r = edges.slot((1ull << 63) | ((uint64_t)(uint32_t)h << 32), &fresh);
    if (fresh) r = add_node(-1, h_hyp_word[h], h, 0);
    int32_t cur = r;
    for (int k = 0; k < len; ++k) {
      const int32_t w = h_phrase_words[o + k];
      int32_t& c = edges.slot(((uint64_t)(uint32_t)cur << 32) | (uint32_t)w, &fresh);
      if (fresh) c = add_node(cur, w, h, k + 1);
      cur = c;
      pair_node[(size_t)o + k] = cur;
    }
    if (len > depth) depth = len;
  }
  f->depth = depth;
  const int32_t n_nodes = (int32_t)parent.size();
  // Levels: level d holds the nodes of depth d-1 that have children, in
  // creation order (a stable bucketing by depth).
  std::vector<int32_t> lv_start((size_t)depth + 1, 0), order;
  for (int32_t i = 0; i < n_nodes; ++i)
    if (ndepth[i] < depth && first_child[i] >= 0) ++lv_start[ndepth[i] + 1];
  for (int d = 0; d < depth; ++d) lv_start[d + 1] += lv_start[d];
  order.resize(lv_start[depth]);
  {
    std::vector<int32_t> fill(lv_start.begin(), lv_start.end() - 1);
    for (int32_t i = 0; i < n_nodes; ++i)
      if (ndepth[i] < depth && first_child[i] >= 0) order[fill[ndepth[i]]++] = i;
  }
  f->rows_lv.resize(depth);
  f->req_lv.resize(depth);
  f->row_base.resize(depth);
  f->req_base.resize(depth);
  f->off_base.resize(depth);
  const int32_t n_rows = lv_start[depth];
  std::vector<int32_t> row(n_nodes, -1), node_req(n_nodes, -1);  // a node's step row; its edge's request
  for (auto* v : {&f->state_row, &f->y_prev, &f->sent}) v->reserve(n_rows);
  f->req_off.reserve((size_t)n_rows + depth);
  f->req.reserve(n_nodes);
  f->req_row.reserve(n_nodes);
  int32_t grow = 0, greq = 0, goff = 0;
  for (int d = 1; d <= depth; ++d) {
    const int32_t b = lv_start[d - 1], e = lv_start[d];
    f->row_base[d - 1] = grow;
    f->req_base[d - 1] = greq;
    f->off_base[d - 1] = goff;
    f->rows_lv[d - 1] = e - b;
    int32_t local = 0;
    for (int32_t i = b; i < e; ++i) {
      const int32_t id = order[i];
      row[id] = grow++;
      f->state_row.push_back(parent[id] < 0 ? hyp[id] : row[parent[id]]);
      f->y_prev.push_back(word[id]);
      f->sent.push_back(h_hyp_sent[hyp[id]]);
      f->req_off.push_back(local);
      for (int32_t c = first_child[id]; c >= 0; c = next_sibling[c]) {
        node_req[c] = greq++;
        f->req.push_back(word[c]);
        f->req_row.push_back(row[id]);
        ++local;
      }
    }
    f->req_off.push_back(local);
    goff += e - b + 1;
    f->req_lv[d - 1] = local;
    if (e - b > f->max_rows) f->max_rows = e - b;
  }
  f->n_rows = grow;
  f->n_req = greq;
  // each pair's path: the request of its edge at every depth
  f->pair_path.assign((size_t)n_pairs * depth, -1);
  for (int p = 0; p < n_pairs; ++p)
    for (int32_t k = 0, o = h_phrase_off[p]; o + k < h_phrase_off[p + 1]; ++k)
      f->pair_path[(size_t)p * depth + k] = node_req[pair_node[(size_t)o + k]];
  f->upload.reserve((size_t)3 * f->n_rows + f->req_off.size() + f->req.size() + f->pair_path.size());
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
  out->pair_of.assign(n, 0);
  out->pair_hyp.clear();
  out->pair_off.assign(1, 0);
  out->pair_words.clear();
  // Open addressing over entry ids, keyed by a hash of (parent, phrase) and
  // confirmed by comparing the words, so equal keys are found whatever the hash.
  size_t cap = 16;
  while (cap < 2 * (size_t)n) cap <<= 1;
  const size_t mask = cap - 1;
  std::vector<int32_t> table(cap, -1);
  std::vector<uint64_t> entry_hash;
  entry_hash.reserve(n);
  for (int32_t j = 0; j < n; ++j) {
    const int32_t o = h_off[j], len = h_off[j + 1] - o;
    uint64_t hv = FlatMap::mix((uint64_t)(uint32_t)h_parent[j] ^ ((uint64_t)len << 32));
    for (int32_t k = 0; k < len; ++k) hv = FlatMap::mix(hv ^ (uint32_t)h_words[o + k]);
    size_t i = hv & mask;
    int32_t found = -1;
    for (; table[i] >= 0; i = (i + 1) & mask) {
      const int32_t p = table[i];
      if (entry_hash[p] != hv || out->pair_hyp[p] != h_parent[j]) continue;
      const int32_t po = out->pair_off[p];
      if (out->pair_off[p + 1] - po != len) continue;
      int32_t k = 0;
      while (k < len && out->pair_words[po + k] == h_words[o + k]) ++k;
      if (k == len) {
        found = p;
        break;
      }
    }
    if (found >= 0) {
      out->pair_of[j] = found;
      continue;
    }
    const int32_t p = (int32_t)out->pair_hyp.size();
    table[i] = p;
    entry_hash.push_back(hv);
    out->pair_of[j] = p;
    out->pair_hyp.push_back(h_parent[j]);
    if (len > 0) out->pair_words.insert(out->pair_words.end(), h_words + o, h_words + o + len);
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
