// Host-only planning of a verification step (no device code): tree
// validation and metadata, the prefix-attention split table, model-shape
// checks and the stochastic acceptance's work list.
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

#include "griffin_verify.h"

namespace griffin_plan {

// Validate one tree against the limits and, where the output pointers are
// non-null, fill depth[n], pos[n] = prefix_len + depth and anc[n] (bit j set
// iff node j is the node or one of its ancestors).  Returns GRIFFIN_OK or the
// status of the first failed check (why, when non-null, gets the message).
int prepare_tree(int32_t n, const int32_t* tokens, const int32_t* parents, int32_t prefix_len, int32_t max_tree,
                 int32_t max_depth, int32_t vocab, int32_t kv_capacity, int32_t* depth, int32_t* pos,
                 uint64_t* anc, std::string* why);

// Prefix-attention work of one step: batch * splits units dealt to the
// sequences by prefix length; tab [batch * splits][4], nsplit [batch].
void attn_split_plan(int batch, const int32_t* prefix_len, const int32_t* n_nodes, int splits, int sp,
                     int32_t* tab, int32_t* nsplit);

// Partial slots the merge reads for a plan: the largest split count of the
// batch rounded up to a power of two (few distinct values, so few captured
// step graphs), at most sp.
int merge_slots(const int32_t* nsplit, int batch, int sp);

// GRIFFIN_OK or GRIFFIN_ESHAPE for a model shape the kernels do not support.
int validate_desc(const griffin_model_desc* d, std::string* why);

// Work list of the stochastic acceptance (rows sorted by child count, the
// k-th child of each row with at least k + 1 children, and its token).
void sampled_plan(int batch, int max_tree, const int32_t* n_nodes, const int32_t* parents,
                  const int32_t* tokens, std::vector<int32_t>& order, std::vector<int>& rows_with,
                  std::vector<int32_t>& step_child, std::vector<int32_t>& step_token);

}  // namespace griffin_plan
