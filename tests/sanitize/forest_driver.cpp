// Drives the host side of ScoreBatch (forest_host.cpp) under the address and
// undefined-behaviour sanitizers: random forests of (hypothesis, phrase)
// pairs, with their structure checked against the phrases, plus every
// argument error of the builder and the predecessor extraction of stack
// rescoring.  Exits non-zero on the first violated check (the sanitizers
// abort on their own findings).
#include <stdio.h>
#include <stdlib.h>

#include <map>
#include <random>
#include <vector>

#include "../../paper_1605_04809_amd/csrc/forest.hpp"

nmt_status nmt::forest_fail(nmt_status st, const char*) { return st; }

#define CHECK(c)                                                   \
  do {                                                             \
    if (!(c)) {                                                    \
      fprintf(stderr, "check failed line %d: %s\n", __LINE__, #c); \
      exit(1);                                                     \
    }                                                              \
  } while (0)

static void check_forest(const nmt_forest* f, int n_hyp, const std::vector<int>& hyp_word,
                         const std::vector<int>& pair_hyp, const std::vector<std::vector<int>>& phr) {
  int32_t depth = 0, n_rows = 0, n_req = 0, max_rows = 0;
  CHECK(nmt_forest_shape(f, &depth, &n_rows, &n_req, &max_rows) == NMT_OK);
  int32_t rows_sum = 0, req_sum = 0;
  std::vector<int32_t> row_level(n_rows, 0), all_state, all_y, all_req_row;
  for (int d = 1; d <= depth; ++d) {
    int32_t R = 0, Q = 0;
    CHECK(nmt_forest_level(f, d, &R, &Q, nullptr, nullptr, nullptr, nullptr, nullptr) == NMT_OK);
    CHECK(R >= 1 && R <= max_rows && Q >= R);
    std::vector<int32_t> st(R), y(R), s(R), off(R + 1), rq(Q);
    CHECK(nmt_forest_level(f, d, nullptr, nullptr, st.data(), y.data(), s.data(), off.data(), rq.data()) == NMT_OK);
    CHECK(off[0] == 0 && off[R] == Q);
    for (int i = 0; i < R; ++i) {
      CHECK(off[i + 1] > off[i]);  // every row has at least one child
      if (d == 1)
        CHECK(st[i] >= 0 && st[i] < n_hyp && y[i] == hyp_word[st[i]]);
      else
        CHECK(st[i] >= 0 && st[i] < rows_sum && row_level[st[i]] == d - 1);
      row_level[rows_sum + i] = d;
      all_state.push_back(st[i]);
      all_y.push_back(y[i]);
      for (int j = off[i]; j < off[i + 1]; ++j) all_req_row.push_back(rows_sum + i);
    }
    rows_sum += R;
    req_sum += Q;
  }
  CHECK(rows_sum == n_rows && req_sum == n_req);
  std::vector<int32_t> path((size_t)phr.size() * depth + 1);
  if (!phr.empty()) CHECK(nmt_forest_pair_paths(f, path.data()) == NMT_OK);
  // each pair walks its phrase: request k asks word k, from the row whose
  // input is word k-1 (the hypothesis' word first) and whose state is the
  // previous request's row
  std::vector<int32_t> all_req;
  for (int d = 1; d <= depth; ++d) {
    int32_t R = 0, Q = 0;
    nmt_forest_level(f, d, &R, &Q, nullptr, nullptr, nullptr, nullptr, nullptr);
    std::vector<int32_t> rq(Q);
    nmt_forest_level(f, d, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, rq.data());
    all_req.insert(all_req.end(), rq.begin(), rq.end());
  }
  for (size_t p = 0; p < phr.size(); ++p)
    for (int k = 0; k < depth; ++k) {
      const int32_t q = path[p * depth + k];
      if (k >= (int)phr[p].size()) {
        CHECK(q == -1);
        continue;
      }
      CHECK(q >= 0 && q < n_req && all_req[q] == phr[p][k]);
      const int32_t row = all_req_row[q];
      CHECK(all_y[row] == (k == 0 ? hyp_word[pair_hyp[p]] : phr[p][k - 1]));
      if (k == 0)
        CHECK(all_state[row] == pair_hyp[p]);
      else
        CHECK(all_state[row] == all_req_row[path[p * depth + k - 1]]);
    }
}

int main() {
  std::mt19937 rng(1234);
  auto U = [&](int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); };
  int forests = 0;
  for (int trial = 0; trial < 300; ++trial) {
    const int n_hyp = U(0, 40), V = U(1, 12);
    std::vector<int> hyp_word(n_hyp), hyp_sent(n_hyp);
    for (int h = 0; h < n_hyp; ++h) {
      hyp_word[h] = U(-1, V - 1);
      hyp_sent[h] = U(0, 3);
    }
    std::vector<int> pair_hyp, off{0}, words;
    std::vector<std::vector<int>> phr;
    const int n_pairs = n_hyp ? U(0, 80) : 0;
    for (int p = 0; p < n_pairs; ++p) {
      pair_hyp.push_back(U(0, n_hyp - 1));
      std::vector<int> w(U(0, 5));
      for (int& x : w) x = U(0, V - 1);
      phr.push_back(w);
      words.insert(words.end(), w.begin(), w.end());
      off.push_back((int)words.size());
    }
    nmt_forest* f = nullptr;
    CHECK(nmt_forest_build(n_hyp, hyp_word.data(), hyp_sent.data(), n_pairs, pair_hyp.data(), off.data(),
                           words.empty() ? nullptr : words.data(), &f) == NMT_OK);
    check_forest(f, n_hyp, hyp_word, pair_hyp, phr);
    // predecessor extraction over the same pairs, repeated twice: duplicates collapse
    std::vector<int> par2(pair_hyp), off2(off), words2(words);
    for (int p = 0; p < n_pairs; ++p) {
      par2.push_back(pair_hyp[p]);
      words2.insert(words2.end(), phr[p].begin(), phr[p].end());
      off2.push_back((int)words2.size());
    }
    nmt::Predecessors P;
    nmt::extract_predecessors(2 * n_pairs, par2.data(), off2.data(), words2.empty() ? nullptr : words2.data(), &P);
    CHECK((int)P.pair_of.size() == 2 * n_pairs && P.pair_off.size() == P.pair_hyp.size() + 1);
    for (int p = 0; p < n_pairs; ++p) {
      CHECK(P.pair_of[p] == P.pair_of[n_pairs + p]);
      const int e = P.pair_of[p];
      CHECK(P.pair_hyp[e] == pair_hyp[p]);
      CHECK(P.pair_off[e + 1] - P.pair_off[e] == (int)phr[p].size());
      for (size_t k = 0; k < phr[p].size(); ++k) CHECK(P.pair_words[P.pair_off[e] + k] == phr[p][k]);
    }
    // distinct pairs stay distinct, numbered in the order of first occurrence
    std::map<std::pair<int, std::vector<int>>, int> first;
    for (int p = 0; p < n_pairs; ++p) first.emplace(std::make_pair(pair_hyp[p], phr[p]), (int)first.size());
    CHECK(P.pair_hyp.size() == first.size());
    for (int p = 0; p < n_pairs; ++p) CHECK(P.pair_of[p] == first.at(std::make_pair(pair_hyp[p], phr[p])));
    nmt_forest_destroy(f);
    ++forests;
  }
  // argument errors
  nmt_forest* f = nullptr;
  int w[2] = {1, 2}, h[2] = {0, 1}, o[3] = {0, 1, 2}, bad_o[3] = {1, 1, 2}, dec_o[3] = {0, 2, 1}, far[2] = {0, 5};
  CHECK(nmt_forest_build(2, w, h, 2, h, o, w, nullptr) == NMT_EINVAL);
  CHECK(nmt_forest_build(-1, w, h, 0, h, o, w, &f) == NMT_EINVAL && !f);
  CHECK(nmt_forest_build(2, nullptr, h, 2, h, o, w, &f) == NMT_EINVAL);
  CHECK(nmt_forest_build(2, w, h, 2, h, bad_o, w, &f) == NMT_EINVAL);
  CHECK(nmt_forest_build(2, w, h, 2, h, dec_o, w, &f) == NMT_EINVAL);
  CHECK(nmt_forest_build(2, w, h, 2, far, o, w, &f) == NMT_ERANGE);
  CHECK(nmt_forest_build(2, w, h, 2, h, o, nullptr, &f) == NMT_EINVAL);
  CHECK(nmt_forest_build(2, w, h, 2, h, o, w, &f) == NMT_OK);
  CHECK(nmt_forest_level(f, 0, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr) == NMT_EINVAL);
  CHECK(nmt_forest_level(f, 2, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr) == NMT_EINVAL);
  CHECK(nmt_forest_pair_paths(f, nullptr) == NMT_EINVAL);
  CHECK(nmt_forest_shape(nullptr, nullptr, nullptr, nullptr, nullptr) == NMT_EINVAL);
  nmt_forest_destroy(f);
  nmt_forest_destroy(nullptr);
  printf("forest driver ok: %d random forests\n", forests);
  return 0;
}
