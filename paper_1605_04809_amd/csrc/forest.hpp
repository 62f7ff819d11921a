// forest.hpp -- host-side data of the ScoreBatch procedure (Section 5.1,
// Figures 1 and 2) and of stack rescoring (Section 5.3, Figure 4), shared by
// forest_host.cpp (plain C++: building the prefix trees, predecessor
// extraction) and forest.hip (the device side).  Not part of the public ABI.
#pragma once

#include <stdint.h>

#include <vector>

#include "../../include/nmt.h"

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

// Sets the calling thread's error message (nmt_last_error) and returns st.
nmt_status forest_fail(nmt_status st, const char* msg);

// The set L of a stack's direct predecessors (Section 5.3): identical
// (parent, phrase) pairs among the n hypotheses of h_parent / h_off /
// h_words are one entry.  pair_of[j] is hypothesis j's entry; entries keep
// the order of their first occurrence, with parents pair_hyp and phrases
// pair_words[pair_off[p] .. pair_off[p+1]).  Arguments are validated by the
// caller.
struct Predecessors {
  std::vector<int32_t> pair_of, pair_hyp, pair_off, pair_words;
};
void extract_predecessors(int32_t n, const int32_t* h_parent, const int32_t* h_off, const int32_t* h_words,
                          Predecessors* out);

// Where each of the n new hypotheses' states comes from after the forest f
// of their predecessors has been scored, then where it goes: plan[j] is the
// forest row that requested hypothesis j's last phrase word, or -(parent+1)
// for an empty phrase (the parent's state is kept); plan[n + j] = first_id + j,
// its row in the state pool.
void gather_plan(const nmt_forest* f, const Predecessors& P, int32_t n, int32_t first_id,
                 std::vector<int32_t>* plan);

}  // namespace nmt
