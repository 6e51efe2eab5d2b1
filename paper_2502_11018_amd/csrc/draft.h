// GRIFFIN-style draft model: arguments and launchers of the kernels around its
// decoder layer (Token-Guided Fusion before it, Token-Enhanced Head after it).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "griffin_internal.h"

namespace griffin {

struct DraftArgs {
  int d, tgf_dim;            // model width, TGF expansion width
  int rows, mpad, max_tree;  // row slots of the step (batch * max_tree), padded to 64
  float ln_eps, rms_eps;
  const uint16_t* embed;     // target's embedding [V][d] (bf16)
  const float* root_feat;    // [batch][d] input feature of each root
  const float* node_feat;    // [rows][d] input feature of every node, or null (then root_feat / feat_r)
  float* feat_r;             // [rows][d] regress features (input of the next pass)
  float* feat_p;             // [rows][d] predict features
  float* h;                  // [mpad][d] TGF fusion h
  float* x;                  // [mpad][d] the decoder layer's residual stream
  const float* parts;        // split-K partials of the current GEMM
  int n_parts_m, n_parts_u, n_parts_d, n_parts_h;
  long long stride_m, stride_u, stride_d, stride_h;  // elements between splits
  uint16_t *x_m, *x_u, *x_d, *x_h, *xn;  // split-bf16 operands of W_m, W_u, W_d, the heads, the LM head
  int ks_m, ks_u, ks_d, ks_h, xn_ks;     // K steps per 64-row tile of each
  const uint16_t *b_m, *ln_h_g, *ln_h_b, *ln_x_g, *ln_x_b, *b_u, *b_d, *b_p, *b_r, *final_norm;  // bf16 [d] / [e]
};

// TGF, stage 0: [F, e] -> x_m; 1: h, [LN(h), LN(e)] -> x_u; 2: SiLU(z) -> x_d;
// 3: o -> x.  Each stage follows the GEMM that fills `parts`.
hipError_t launch_draft_front(const DraftArgs& a, const StepMeta& meta, int stage, hipStream_t s);
// TEH, stage 0: y = x + layer residual -> x_h; 1: F^R -> feat_r, RMSNorm(F^P) -> xn.
hipError_t launch_draft_head(const DraftArgs& a, const StepMeta& meta, const ResidualAdd& add, int stage,
                             hipStream_t s);
// Top-k (k <= 16) tokens and log-probabilities of every live row of logits
// [rows][ld] (V <= 524288); `work` holds draft_topk_work_bytes(rows, V).
size_t draft_topk_work_bytes(int rows, int V);
hipError_t launch_draft_topk(const float* logits, long long ld, int V, const StepMeta& meta, int rows, int max_tree,
                             int k, int32_t* tok, float* logp, float* work, hipStream_t s);

}  // namespace griffin

namespace griffin {

// Device-side expansion of a draft tree (Sec. 3.1, the EAGLE-2 style dynamic
// tree the draft builds): after pass t's top-k, one workgroup per sequence
// scores the candidates of the pass's frontier, and either writes the next
// pass tree (the k best of them, appended to the pass tree in the step
// metadata, plus the next pass's fixed metadata) or, after the last pass,
// selects the n_total best of all candidates.  Candidate scores are fp64
// sums of fp32 log-probabilities, ranked by score (NaN lowest), ties to the
// earlier candidate.
constexpr int DRAFT_SEL_MAX = 1024;  // candidates per sequence: k (1 + k (depth - 1)) <= 16 * 64
struct DraftSelectArgs {
  int t, k, depth, n_total, max_tree;
  const int32_t* topk_tok;  // [batch * max_tree][k] of pass t
  const float* topk_lp;
  int32_t* c_tok;           // [batch][DRAFT_SEL_MAX] candidates: token, proposing pass-tree node, score
  int32_t* c_node;
  double* c_score;
  int32_t* n_cand;          // [batch * max_tree] pass-tree node -> its candidate
  double* n_score;          // [batch * max_tree] pass-tree node -> its score
  int32_t* m_token;         // the step metadata's tree rows [batch * max_tree]
  int32_t* m_parent;
  uint64_t* m_anc;
  const uint4* tail_src;    // next pass's fixed metadata (prefix, sizes, positions, depths, split table)
  uint4* tail_dst;
  int tail_words;
  int32_t* o_nodes;         // last pass: [batch] node counts, [batch][max_tree] tokens, parents, scores
  int32_t* o_tok;
  int32_t* o_par;
  float* o_score;
};
hipError_t launch_draft_select(const DraftSelectArgs& a, int batch, hipStream_t s);

}  // namespace griffin
