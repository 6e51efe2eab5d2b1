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
