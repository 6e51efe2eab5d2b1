// Stochastic (temperature > 0) tree acceptance: the launcher and its scratch.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace griffin {

// Stochastic acceptance (temperature > 0): every node's rejection chain
// advances one child per launch, the vocabulary spread over workgroups.
struct SampledArgs {
  const int32_t* n_nodes;   // [B]
  const int32_t* token;     // [B][max_tree]
  const int32_t* parent;    // [B][max_tree] (the root's entry is not read)
  const float* logits;      // [B][max_tree][vocab] target logits at every node
  const float* q;           // [B][max_tree][vocab] draft distribution of each node's children
  const float* u_accept;    // [B][max_tree] uniform for the test at each child
  const float* u_final;     // [B][max_tree] uniform for the token drawn at each node
  const int32_t* order;     // rows b * max_tree + u of every node, by child count, descending
  const int32_t* step_child;  // for k = 0, 1, ..: the k-th child (node id) of each of the first
  const int32_t* step_token;  // rows_with[k + 1] rows of `order`, and its token
  void* scratch;             // sampled_scratch_bytes(scratch_batch, max_tree, vocab)
  int32_t* result;          // [B][result_stride(max_depth)]: L, NaN flag, L + 1 tokens, L path nodes
  float inv_t;              // 1 / temperature
  int batch, scratch_batch, max_tree, max_depth, vocab;
};

int sampled_nslice(int vocab);
size_t sampled_scratch_bytes(int batch, int max_tree, int vocab);
// rows_with[j] = rows of `order` with >= j children (j = 0 .. max_children,
// rows_with[0] = all nodes).
hipError_t launch_sampled_accept(const SampledArgs& a, const int* rows_with, int max_children, hipStream_t s);

// The current device's copy of the library's fixed scratch block (a
// file-scope device array of kStaticScratchBytes, looked up once per device):
// *ptr is its device address, *bytes its size.
constexpr size_t kStaticScratchBytes = 4u << 20;
hipError_t static_scratch(void** ptr, size_t* bytes);

}  // namespace griffin
