// Host-only planning of a verification step: tree validation and metadata,
// the prefix-attention split table, the model-shape checks and the work list
// of the stochastic acceptance.  Plain C++ with no device code, so it also
// builds into a CPU test program under the address and undefined-behaviour
// sanitizers.

#include "plan.h"

#include <algorithm>
#include <cstdio>

namespace griffin_plan {

constexpr int kMaxTree = 64;

// Validate one tree and, optionally, fill depth / position / ancestor masks.
int prepare_tree(int32_t n, const int32_t* tokens, const int32_t* parents, int32_t prefix_len, int32_t max_tree,
                 int32_t max_depth, int32_t vocab, int32_t kv_capacity, int32_t* depth, int32_t* pos,
                 uint64_t* anc, std::string* why) {
  auto fail = [&](int code, const char* fmt, long a = 0, long b = 0) {
    if (why) {
      char buf[256];
      snprintf(buf, sizeof buf, fmt, a, b);
      *why = buf;
    }
    return code;
  };
  if (!tokens || !parents) return fail(GRIFFIN_EINVAL, "null tree array");
  if (n < 1 || n > max_tree || n > kMaxTree) return fail(GRIFFIN_ETREE, "tree size %ld outside [1, %ld]", n, max_tree);
  if (prefix_len < 0 || (long)prefix_len + n > kv_capacity)
    return fail(GRIFFIN_ECAPACITY, "prefix_len %ld + nodes %ld exceeds kv_capacity", prefix_len, n);
  if (parents[0] != -1) return fail(GRIFFIN_ETREE, "parents[0] = %ld, must be -1", parents[0]);
  int32_t dep[kMaxTree];
  uint64_t an[kMaxTree];
  dep[0] = 0;
  an[0] = 1ull;
  for (int i = 0; i < n; ++i) {
    if (tokens[i] < 0 || tokens[i] >= vocab) return fail(GRIFFIN_ETOKEN, "token %ld of node %ld out of range", tokens[i], i);
    if (i == 0) continue;
    const int p = parents[i];
    if (p < 0 || p >= i) return fail(GRIFFIN_ETREE, "parent %ld of node %ld not in [0, i)", p, i);
    dep[i] = dep[p] + 1;
    if (dep[i] > max_depth) return fail(GRIFFIN_ETREE, "node %ld has depth %ld > max_depth", i, dep[i]);
    an[i] = an[p] | (1ull << i);
  }
  for (int i = 0; i < n; ++i) {
    if (depth) depth[i] = dep[i];
    if (pos) pos[i] = prefix_len + dep[i];
    if (anc) anc[i] = an[i];
  }
  return GRIFFIN_OK;
}

// Prefix-attention work of one step: batch * splits units, each sequence at
// least one and at most min(sp, blocks / 2) (blocks = 32-key blocks of its
// prefix), the rest dealt one at a time to the sequence with the most blocks
// per split (ties: the lower index).  A sequence's result depends on the
// batch only through its split count.  tab [batch * splits][4]: (b | split <<
// 16, splits of b, prefix_len, n_nodes), b = -1 for units left unused;
// nsplit [batch].
void attn_split_plan(int batch, const int32_t* prefix_len, const int32_t* n_nodes, int splits, int sp,
                     int32_t* tab, int32_t* nsplit) {
  std::vector<int> blocks(batch), cap(batch), cnt(batch, 1);
  for (int b = 0; b < batch; ++b) {
    blocks[b] = (prefix_len[b] + 31) / 32;
    cap[b] = std::max(1, std::min(sp, blocks[b] / 2));
  }
  for (int left = batch * splits - batch; left > 0; --left) {
    int best = -1;
    for (int b = 0; b < batch; ++b)
      if (cnt[b] < cap[b] && (best < 0 || (long long)blocks[b] * cnt[best] > (long long)blocks[best] * cnt[b]))
        best = b;
    if (best < 0) break;
    ++cnt[best];
  }
  int j = 0;
  for (int b = 0; b < batch; ++b) {
    nsplit[b] = cnt[b];
    for (int s = 0; s < cnt[b]; ++s, ++j) {
      tab[4 * j] = b | (s << 16);
      tab[4 * j + 1] = cnt[b];
      tab[4 * j + 2] = prefix_len[b];
      tab[4 * j + 3] = n_nodes[b];
    }
  }
  for (; j < batch * splits; ++j) {
    tab[4 * j] = -1;
    tab[4 * j + 1] = tab[4 * j + 2] = tab[4 * j + 3] = 0;
  }
}

int merge_slots(const int32_t* nsplit, int batch, int sp) {
  int most = 1;
  for (int b = 0; b < batch; ++b) most = std::max(most, (int)nsplit[b]);
  int slots = 1;
  while (slots < most) slots *= 2;
  return std::min(slots, sp);
}

int validate_desc(const griffin_model_desc* d, std::string* why) {
  auto bad = [&](const char* m) {
    if (why) *why = m;
    return GRIFFIN_ESHAPE;
  };
  if (d->n_layers < 1 || d->d_model < 8 || d->vocab < 2 || d->d_ff < 8) return bad("non-positive dimension");
  if (d->head_dim != 64 && d->head_dim != 128) return bad("head_dim must be 64 or 128");
  if (d->n_kv_heads < 1 || d->n_q_heads < 1 || d->n_q_heads % d->n_kv_heads) return bad("n_q_heads must be a multiple of n_kv_heads");
  if (d->d_model % 8 || d->d_ff % 8 || (d->n_q_heads * d->head_dim) % 8) return bad("d_model, d_ff, n_q_heads*head_dim must be multiples of 8");
  if (d->d_model > 8192) return bad("d_model above 8192");
  if (d->n_experts < 1 || d->n_experts > 64) return bad("n_experts must be in [1, 64]");
  if (d->n_experts > 1 && (d->top_k < 1 || d->top_k > 4 || d->top_k > d->n_experts)) return bad("top_k must be in [1, min(n_experts, 4)]");
  if (d->max_batch < 1) return bad("max_batch < 1");
  if (d->max_tree < 1 || d->max_tree > kMaxTree) return bad("max_tree must be in [1, 64]");
  if (d->max_depth < 0 || d->max_depth >= d->max_tree) return bad("max_depth must be in [0, max_tree - 1]");
  if (d->kv_capacity < 32 || d->kv_capacity % 32) return bad("kv_capacity must be a positive multiple of 32");
  if (!(d->rms_eps > 0.f) || !(d->rope_base > 1.0)) return bad("rms_eps must be > 0 and rope_base > 1");
  return GRIFFIN_OK;
}

// Work list of the stochastic acceptance: every node's row b * max_tree + u,
// sorted by child count (descending, ties by row); rows_with[j] = the number
// of rows with at least j children; for k = 0, 1, .. in turn, the k-th child
// (in id order) of each of the first rows_with[k + 1] rows and its token.
// parents: root entries ignored.
void sampled_plan(int batch, int max_tree, const int32_t* n_nodes, const int32_t* parents,
                         const int32_t* tokens, std::vector<int32_t>& order, std::vector<int>& rows_with,
                         std::vector<int32_t>& step_child, std::vector<int32_t>& step_token) {
  std::vector<std::vector<int32_t>> kids((size_t)batch * max_tree);
  order.clear();
  for (int b = 0; b < batch; ++b)
    for (int i = 0; i < n_nodes[b]; ++i) {
      order.push_back(b * max_tree + i);
      if (i > 0) kids[(size_t)b * max_tree + parents[(size_t)b * max_tree + i]].push_back(i);
    }
  std::stable_sort(order.begin(), order.end(),
                   [&](int32_t x, int32_t y) { return kids[x].size() > kids[y].size(); });
  const int cmax = order.empty() ? 0 : (int)kids[order[0]].size();
  rows_with.assign(cmax + 1, 0);
  for (int32_t r : order)
    for (int j = 0; j <= (int)kids[r].size(); ++j) ++rows_with[j];
  step_child.clear();
  step_token.clear();
  for (int k = 0; k < cmax; ++k)
    for (int i = 0; i < rows_with[k + 1]; ++i) {
      const int32_t r = order[i], c = kids[r][k];
      step_child.push_back(c);
      step_token.push_back(tokens[(size_t)(r / max_tree) * max_tree + c]);
    }
}

}  // namespace griffin_plan
