/*
 * griffin_verify.h - tree verification for GRIFFIN-style speculative decoding
 * on one AMD Instinct MI355X (gfx950).
 *
 * What the library computes.  In each draft-and-verify cycle the target model
 * scores every draft token in a single forward pass (paper, Sec. 3).  The draft
 * tokens form a tree because several top-k candidates are kept per position
 * (Sec. 4.1), and a draft token counts only if the target's own greedy
 * prediction at its parent equals it, a rejection discarding everything below
 * it (Sec. 4.1); decoding is greedy at temperature 0 (Sec. 5).  The library
 * therefore takes a prefix KV cache plus a draft tree per sequence and returns
 * the greedy acceptance length and the accepted tokens: the deepest node whose
 * whole root path is accepted, then the target's prediction at that node (the
 * extra token the paper's acceptance length counts, Sec. 5).  Trees follow the
 * paper's appendix "Draft Tree Structure" (up to 64 nodes here; the paper uses
 * 60 draft tokens at depth 6).
 *
 * Conventions shared by every entry point.
 *  - A tree has n nodes; node 0 is the root: the last accepted token, which is
 *    not yet in the KV cache.  parents[0] = -1 and 0 <= parents[i] < i.
 *  - Node i sits at sequence position prefix_len + depth(i) (rotary position)
 *    and its K/V go to cache slot prefix_len + i.  Slots [prefix_len,
 *    prefix_len + n) are scratch: each step overwrites them.  For a chain
 *    (parents[i] = i - 1) slot and position coincide, so committing a chain is
 *    just prefix_len += n.
 *  - The model is a LLaMA-family decoder (RMSNorm, rotate-half rotary
 *    embedding, grouped-query attention with contiguous groups, SwiGLU MLP) or
 *    its Mixtral mixture-of-experts variant (softmax router, top-k experts,
 *    kept probabilities renormalised); these are the targets of Sec. 5.
 *  - Greedy argmax ties go to the lowest token id; among equally deep accepted
 *    nodes the one with the smallest id is reported.
 *  - bf16 means IEEE bfloat16 bit patterns (uint16).  All device pointers are
 *    borrowed: the caller allocates them, keeps them alive while the context
 *    lives, and frees them.  Device pointers must be 16-byte aligned.
 *  - Every function returns GRIFFIN_OK (0) or a negative status; argument and
 *    tree validation happens before any device work, so on a validation error
 *    nothing is launched and nothing (KV cache included) is written.
 *  - A context is not thread-safe.  Several contexts may borrow the same
 *    weights; two contexts must not share a KV cache region they both write.
 */
#ifndef GRIFFIN_VERIFY_H
#define GRIFFIN_VERIFY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GRIFFIN_OK 0
#define GRIFFIN_EINVAL (-1)    /* null or inconsistent argument */
#define GRIFFIN_ESHAPE (-2)    /* model shape the kernels do not support */
#define GRIFFIN_ETREE (-3)     /* malformed tree: parents[0] != -1, parent not in [0,i), n out of [1,max_tree], depth > max_depth */
#define GRIFFIN_ETOKEN (-4)    /* token id outside [0, vocab) */
#define GRIFFIN_ECAPACITY (-5) /* prefix_len < 0 or prefix_len + n > kv_capacity */
#define GRIFFIN_EORDER (-6)    /* griffin_accept / griffin_read_predictions / griffin_read_features before any step */
#define GRIFFIN_ENOMEM (-7)    /* device or pinned host allocation failed */
#define GRIFFIN_EHIP (-8)      /* a HIP runtime call failed; griffin_last_error has the text */
#define GRIFFIN_ENUMERIC (-9)  /* a NaN appeared in the logits of a valid tree node */

/* Model shape and limits.  Supported: head_dim 64 or 128; n_q_heads a
 * multiple of n_kv_heads; d_model, n_q_heads*head_dim and d_ff multiples of 8;
 * n_experts in [1, 64] with top_k in [1, min(n_experts, 4)] when n_experts > 1;
 * max_tree in [1, 64]; max_depth in [0, max_tree - 1]; kv_capacity a positive
 * multiple of 32. */
typedef struct griffin_model_desc {
  int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ff, vocab;
  int32_t n_experts; /* 1 = dense SwiGLU MLP */
  int32_t top_k;     /* experts per token when n_experts > 1 (ignored otherwise) */
  float rms_eps;
  double rope_base;
  int32_t max_batch;   /* sequences per step */
  int32_t max_tree;    /* nodes per tree, root included (<= 64) */
  int32_t max_depth;   /* deepest node depth accepted by the validator */
  int32_t kv_capacity; /* cache slots per (layer, sequence, KV head) */
} griffin_model_desc;

/* Device weights, bf16, row-major.  Per-layer fields point to host arrays of
 * n_layers device pointers (the host arrays are copied at init).
 * The projection matrices (w_qkv, w_o, w_gate_up, w_down) and lm_head are read
 * only by griffin_verify_init, which repacks them into a buffer the context
 * owns (same size as the originals); the caller may free them after init.
 * embed, the norm gains and w_router are borrowed for the context's lifetime.
 *   embed       [vocab][d_model]
 *   lm_head     [vocab][d_model]          (untied)
 *   final_norm  [d_model]
 *   attn_norm   [d_model]                 RMSNorm gain before attention
 *   w_qkv       [(Hq + 2*Hkv)*head_dim][d_model]; rows are all query heads,
 *               then all key heads, then all value heads (head-major)
 *   w_o         [d_model][Hq*head_dim]
 *   mlp_norm    [d_model]
 *   w_gate_up   dense: [2*d_ff][d_model] (gate rows, then up rows)
 *               MoE:   [n_experts][2*d_ff][d_model]
 *   w_down      dense: [d_model][d_ff];  MoE: [n_experts][d_model][d_ff]
 *   w_router    MoE: [n_experts][d_model]; NULL (the array itself) for dense */
typedef struct griffin_weights {
  const void *embed, *lm_head, *final_norm;
  const void *const *attn_norm, *const *w_qkv, *const *w_o, *const *mlp_norm;
  const void *const *w_gate_up, *const *w_down, *const *w_router;
} griffin_weights;

typedef struct griffin_ctx griffin_ctx;

/* Bytes of one of the two KV cache buffers for this shape:
 * n_layers * max_batch * n_kv_heads * kv_capacity * head_dim * 2. */
size_t griffin_kv_cache_bytes(const griffin_model_desc *desc);

/* Create a context.
 * k_cache: device bf16 [n_layers][max_batch][n_kv_heads][kv_capacity][head_dim],
 *          keys after rotation.
 * v_cache: device bf16 [n_layers][max_batch][n_kv_heads][kv_capacity/32][head_dim][32]
 *          (values in 32-slot tiles, each stored transposed: slot s of a
 *          head, dimension j lives at tile s/32, row j, column s%32).
 * hip_stream: the hipStream_t every launch is enqueued on (NULL = default).
 * The context allocates its own workspace (the repacked weights, activations,
 * partial sums, metadata, pinned staging) and frees it in griffin_verify_free;
 * init synchronises the stream once the repacking is done.
 * Errors: EINVAL (null pointer, misaligned pointer), ESHAPE, ENOMEM, EHIP. */
int griffin_verify_init(const griffin_model_desc *desc, const griffin_weights *weights,
                        void *k_cache, void *v_cache, void *hip_stream, griffin_ctx **out);

/* Enqueue one verification pass over `batch` trees (asynchronous).
 * Host arrays, row b of each describes sequence b (cache row b):
 *   prefix_len [batch]            cached positions of sequence b
 *   n_nodes    [batch]            tree size, root included
 *   tokens     [batch][max_tree]  token of node i (entries >= n_nodes ignored)
 *   parents    [batch][max_tree]  parent of node i; parents[b][0] = -1
 * logits_out: optional device fp32 [batch*max_tree][vocab]; row b*max_tree+i
 *   receives node i's logits (rows of absent nodes are left untouched).
 * The pass writes the trees' K/V into cache slots [prefix_len, prefix_len+n)
 * of each sequence, then runs the acceptance walk on the device.  The host
 * arrays may be reused as soon as the call returns.
 * Errors: EINVAL, ETREE, ETOKEN, ECAPACITY (nothing launched), EHIP. */
int griffin_verify_step(griffin_ctx *ctx, int32_t batch, const int32_t *prefix_len,
                        const int32_t *n_nodes, const int32_t *tokens, const int32_t *parents,
                        float *logits_out);

/* Wait for the last step and copy its acceptance result to host arrays:
 *   accept_len [batch]                 accepted draft tokens L in [0, max_depth]
 *   tokens_out [batch][max_depth + 1]  L accepted tokens, then the target's
 *                                      prediction at the last accepted node;
 *                                      remaining entries -1
 *   path_nodes [batch][max_depth]      node ids of the accepted tokens, -1 padded
 * Any output pointer may be NULL.  The paper's acceptance length is L + 1.
 * Errors: EORDER (no step yet), EHIP, ENUMERIC (a NaN logit in a valid node;
 * the outputs are still written). */
int griffin_accept(griffin_ctx *ctx, int32_t *accept_len, int32_t *tokens_out, int32_t *path_nodes);

/* Stochastic acceptance of the last step's trees at temperature T > 0 (the
 * paper evaluates T = 1 beside greedy decoding, Sec. 5, and relies on the
 * method being lossless).  Recursive rejection sampling over each node's
 * children, in node-id order; the children of node u must have been drawn
 * from u's draft distribution q_u without replacement:
 *   p = softmax(logits_u / T), q = q_u;
 *   child with token t: accepted when u_accept[child] < min(1, p(t) / q(t));
 *   otherwise p <- max(p - q, 0) renormalised and t leaves q (renormalised);
 *   a child accepted: continue there; none accepted, or no children: emit one
 *   token drawn from p with u_final[u] (the first token whose cumulative sum
 *   exceeds u_final * sum, in token order).
 * Degenerate inputs: q(t) = 0 accepts when p(t) > 0; a residual summing to
 * zero leaves p unchanged.
 *   logits    device fp32 [batch*max_tree][vocab]: the buffer the last
 *             griffin_verify_step filled (logits_out must have been given)
 *   q_draft   device fp32 [batch*max_tree][vocab]: row b*max_tree+u = the
 *             draft distribution u's children were drawn from (finite, >= 0,
 *             any positive scale; rows of leaves are not read); or NULL for a
 *             deterministic draft, such as the top-k expansion of
 *             griffin_draft_tree (App. "Draft Tree Structure"), whose children
 *             are a function of the draft rather than draws from it: each
 *             child is then the point mass at its own token, accepted with
 *             probability p(t) / D (D = mass of p left after the node's
 *             earlier rejections), and a rejection removes t from p (nothing
 *             for a token already removed, or when no mass would be left).
 *             Lossless for any such tree.
 *   u_accept  host [batch][max_tree], u_final host [batch][max_tree]:
 *             uniform draws in [0, 1) (entries of absent nodes are checked
 *             but not used)
 * Outputs as for griffin_accept: L accepted draft tokens, then the emitted
 * token.  Synchronises the context's stream.  Errors: EINVAL (NULL logits or
 * uniforms, T <= 0 or not finite, a uniform outside [0, 1)), EORDER (no step yet),
 * EHIP, ENUMERIC (a NaN logit at a node the walk visited). */
int griffin_accept_sampled(griffin_ctx *ctx, const float *logits, const float *q_draft,
                           const float *u_accept, const float *u_final, float temperature,
                           int32_t *accept_len, int32_t *tokens_out, int32_t *path_nodes);

/* Commit the accepted path of the last step into the KV cache (asynchronous,
 * on the context's stream).  The path is the one the last acceptance call
 * since that step returned: griffin_accept (greedy) or griffin_accept_sampled
 * (temperature > 0), whichever ran last.  For every sequence b of that step,
 * with L accepted draft nodes n_1..n_L at depths 1..L: their K/V,
 * already rotated at positions prefix_len + k, move from scratch slots
 * prefix_len + n_k to slots prefix_len + k, so that slots [0, prefix_len + L]
 * hold the plain causal cache of prefix + root + accepted tokens.  The caller
 * continues with prefix_len + L + 1 and the target's extra token (tokens_out
 * entry L of the acceptance call) as the next root.  The paper's
 * losslessness: a loop of step / accept / commit emits exactly the target's
 * greedy tokens (and, with griffin_accept_sampled, samples of the target's
 * distribution).
 * Errors: EINVAL, EORDER (no step yet, or no acceptance call since the last
 * step), EHIP. */
int griffin_commit(griffin_ctx *ctx);

/* Wait for the last step and copy the target's greedy prediction (argmax of
 * the logits) of every node: pred [batch][max_tree] host, -1 for absent nodes.
 * Errors: EORDER, EHIP. */
int griffin_read_predictions(griffin_ctx *ctx, int32_t *pred);

/* Wait for the last step and copy every node's top-2 logit margin: the
 * largest logit minus the second largest (0 when the largest value occurs
 * twice), over the non-NaN entries of the node's row: margin [batch][max_tree]
 * host fp32, -1 for absent nodes, NaN for a row with fewer than two non-NaN
 * logits.  A greedy choice whose margin is within the logits' rounding error
 * is a near tie (Sec. 5: greedy decoding is decided by the argmax alone).
 * Errors: EORDER, EHIP. */
int griffin_read_margins(griffin_ctx *ctx, float *margin);

/* Mixture-of-experts models only (the Mixtral targets of Sec. 5): wait for
 * the last step and copy the fp32 router logits its pass computed, before the
 * softmax and top-k, for every layer and node: out [n_layers][batch][max_tree]
 * [n_experts] host, zeros for absent nodes.  A diagnostic of the routing
 * decisions (a near tie between the last kept and first dropped expert is
 * where a rounding difference can change a token's experts).
 * Errors: EINVAL (dense model), EORDER (no step yet), EHIP. */
int griffin_read_router_logits(griffin_ctx *ctx, float *out);

/* The target's features of chosen nodes of the last step: the hidden state
 * after the last layer, before the final norm, i.e. the feature that
 * EAGLE-style drafting predicts and feeds back (Sec. 3; the draft of Sec. 4.2
 * takes the feature of the token before each input token).  nodes host
 * [batch][n], node ids of that step's trees, -1 for a zero row; out device
 * fp32 [batch][n][d_model], written in stream order after the step (valid
 * until the next step; no synchronisation).  1 <= batch <= the step's batch,
 * 1 <= n <= max_tree.  Errors: EINVAL, EORDER (no step yet), ETREE (a node
 * that is not in its sequence's tree), EHIP. */
int griffin_read_features(griffin_ctx *ctx, int32_t batch, int32_t n, const int32_t *nodes, float *out);

/* Replay the launch sequence of a step from a captured HIP graph (default:
 * enabled).  One graph is captured per (batch, logits_out) pair on its first
 * step and replayed afterwards (at most 8 are kept, the oldest is dropped);
 * every per-step input travels through device buffers whose addresses are
 * fixed for the context, so replays compute exactly what plain launches do.
 * Steps use plain launches while per-class timing is enabled or when the
 * context was created on the legacy null stream.  enable: 0 = plain launches.
 * Errors: EINVAL (null context). */
int griffin_set_graphs(griffin_ctx *ctx, int32_t enable);

/* Precision of the GEMM operands.  Default (bf16_only = 0): each activation
 * enters the projections as a bf16 high part plus a bf16 low part, two MFMAs
 * per weight fragment, which keeps fp32-grade activations against bf16
 * weights.  bf16_only = 1: the high part alone, i.e. activations rounded to
 * bf16 as in a plain bf16 forward pass (the paper's setting), half the
 * activation staging and MFMA work per weight byte.  Weights are bf16 either
 * way; norms, RoPE, attention and reductions are unchanged.  Waits for the
 * stream and drops captured graphs.  Errors: EINVAL, EHIP. */
int griffin_set_activation_precision(griffin_ctx *ctx, int32_t bf16_only);

/* Release the context (waits for its stream first).  NULL is a no-op. */
void griffin_verify_free(griffin_ctx *ctx);

/* Static text for a status code. */
const char *griffin_status_str(int code);

/* Text of the last error recorded on ctx ("" if none). */
const char *griffin_last_error(const griffin_ctx *ctx);

/* Host-only tree validation and metadata (no device work, no context).
 * For one tree of n nodes: checks it like griffin_verify_step does against
 * (max_tree, max_depth, vocab, kv_capacity) and fills, when non-NULL,
 *   depth [n]    node depth (root 0)
 *   pos   [n]    prefix_len + depth (rotary position)
 *   anc   [n]    bit j set iff node j is node i or one of its ancestors
 * Errors: EINVAL, ETREE, ETOKEN, ECAPACITY. */
int griffin_tree_prepare(int32_t n, const int32_t *tokens, const int32_t *parents, int32_t prefix_len,
                         int32_t max_tree, int32_t max_depth, int32_t vocab, int32_t kv_capacity,
                         int32_t *depth, int32_t *pos, uint64_t *anc);

/* Run only the device acceptance walk on given predictions (no model, no
 * context): for `batch` trees (host arrays laid out as in griffin_verify_step)
 * and host pred [batch][max_tree] (the target's prediction per node), fill the
 * same outputs as griffin_accept.  Allocates and frees its own device buffers
 * and synchronises hip_stream.  Errors: EINVAL, ETREE, ETOKEN, ENOMEM, EHIP. */
int griffin_accept_walk(void *hip_stream, int32_t batch, int32_t max_tree, int32_t max_depth,
                        int32_t vocab, const int32_t *n_nodes, const int32_t *tokens,
                        const int32_t *parents, const int32_t *pred, int32_t *accept_len,
                        int32_t *tokens_out, int32_t *path_nodes);

/* The stochastic acceptance of griffin_accept_sampled for trees given
 * directly: n_nodes, tokens, parents and the uniforms are host arrays laid
 * out as for griffin_verify_step / griffin_accept_sampled; logits and q_draft
 * are device fp32 [batch*max_tree][vocab] (q_draft NULL: a deterministic
 * draft, as for griffin_accept_sampled).  Allocates and frees its own
 * device buffers and synchronises hip_stream.  Errors: EINVAL, ETREE, ETOKEN,
 * ENOMEM, EHIP, ENUMERIC (outputs still written). */
int griffin_accept_sampled_walk(void *hip_stream, int32_t batch, int32_t max_tree, int32_t max_depth,
                                int32_t vocab, const int32_t *n_nodes, const int32_t *tokens,
                                const int32_t *parents, const float *logits, const float *q_draft,
                                const float *u_accept, const float *u_final, float temperature,
                                int32_t *accept_len, int32_t *tokens_out, int32_t *path_nodes);

/* griffin_accept_sampled_walk without any device allocation, for callers that
 * cannot allocate (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, same kernels and the
 * same results as griffin_accept_sampled_walk.  Its device memory (the
 * staged tree and uniforms, the kernels' scratch and the result) is a fixed
 * 4 MiB block (4194304 bytes) that the library holds on every GPU it runs on
 * until the process ends; a call needs
 *   4 * (7 * batch * max_tree + batch) + sampled scratch + 4 * batch * (3 + 2 * max_depth) + 768
 * bytes, the sampled scratch being about 1.3 MB for batch 8, max_tree 64,
 * vocab 128256 (about 24 such sequences fit).  Calls that need more return
 * GRIFFIN_ENOMEM before any device work.  Every call on one GPU shares that
 * GPU's block: calls that overlap in time on the same GPU (two host threads,
 * or two streams whose work interleaves) race and must be serialised by the
 * caller.  The block keeps the last call's contents; the kernels read nothing
 * they have not written in the same call.  Host-side bookkeeping uses
 * ordinary host memory.  Synchronises hip_stream.
 * Errors: EINVAL, ETREE, ETOKEN, ENOMEM (beyond the fixed block), EHIP,
 * ENUMERIC (outputs still written). */
int griffin_accept_sampled_walk_noalloc(void *hip_stream, int32_t batch, int32_t max_tree, int32_t max_depth,
                                        int32_t vocab, const int32_t *n_nodes, const int32_t *tokens,
                                        const int32_t *parents, const float *logits, const float *q_draft,
                                        const float *u_accept, const float *u_final, float temperature,
                                        int32_t *accept_len, int32_t *tokens_out, int32_t *path_nodes);

/* ------------------------------------------------------------ draft model
 * A GRIFFIN-style draft model (Sec. 4.2): Token-Guided Fusion of an input
 * feature F and the token embedding e,
 *   h = [F, e] W_m + b_m,  z = [LN(h), LN(e)] W_u + b_u,  o = SiLU(z) W_d + b_d + h,
 * one decoder layer of the target's shape over o (rotary attention over the
 * draft's own cache of the prefix and the node's ancestors in the draft
 * tree), and the Token-Enhanced Head, two heads on the layer output y:
 * the predict feature F^P = y W_p + b_p, mapped to tokens by the target's final
 * norm and LM head, and the regress feature F^R = y W_r + b_r, the input
 * feature of the node's children in the next draft pass.  LN is LayerNorm
 * with gain and bias.  The paper gives no equations for the decoder layer and
 * the heads; the library takes these readings. */
typedef struct griffin_draft griffin_draft;

/* Device bf16 tensors of a draft model, row-major [out][in]:
 *   w_m [d][2d], b_m [d]; ln_h_g, ln_h_b, ln_x_g, ln_x_b [d];
 *   w_u [tgf_dim][2d], b_u [tgf_dim]; w_d [d][tgf_dim], b_d [d];
 *   w_p, w_r [d][d], b_p, b_r [d];
 *   the decoder layer as in griffin_weights (one layer, dense).
 * The matrices are repacked at init (the caller may free them afterwards);
 * biases, LayerNorm parameters and norm gains are borrowed. */
typedef struct griffin_draft_weights {
  const void *w_m, *b_m, *ln_h_g, *ln_h_b, *ln_x_g, *ln_x_b, *w_u, *b_u, *w_d, *b_d;
  const void *w_p, *b_p, *w_r, *b_r;
  const void *attn_norm, *w_qkv, *w_o, *mlp_norm, *w_gate_up, *w_down;
} griffin_draft_weights;

/* Create a draft context.  desc: the target's shape (its n_layers is ignored:
 * the draft has one layer; n_experts must be 1; vocab at most 524288;
 * d_model at most 8192) with the draft's own limits: max_batch, max_tree
 * (>= 1 + k * (depth - 1) expanded nodes and >= n_total + 1 drafted nodes),
 * max_depth (>= depth - 1), kv_capacity.  embed, lm_head,
 * final_norm: the target's (embed and final_norm borrowed, lm_head repacked).
 * k_cache, v_cache: the draft layer's cache, laid out as for
 * griffin_verify_init with one layer (prefix K/V of the draft layer).
 * Errors: EINVAL, ESHAPE, ENOMEM, EHIP. */
int griffin_draft_init(const griffin_model_desc *desc, int32_t tgf_dim, float ln_eps,
                       const griffin_draft_weights *weights, const void *embed, const void *lm_head,
                       const void *final_norm, void *k_cache, void *v_cache, void *hip_stream,
                       griffin_draft **out);
void griffin_draft_free(griffin_draft *draft);

/* The draft's one-layer verify context (for griffin_write_prefix-style cache
 * set-up, timing and error strings: griffin_last_error(griffin_draft_context(d))). */
griffin_ctx *griffin_draft_context(griffin_draft *draft);

/* One draft pass over `batch` trees laid out as for griffin_verify_step
 * (node 0 the root at position prefix_len; a node's input feature is its
 * parent's regress feature from the previous pass, the root's is
 * root_features, device fp32 [batch][d]).  Writes, per node row
 * b * max_tree + i, its k most probable next tokens (value descending, lower
 * id first on ties) and their log-probabilities: host topk_tokens, topk_logp
 * [batch * max_tree][k], 1 <= k <= 16 (rows of absent nodes untouched).
 * Synchronises the stream.  Errors as griffin_verify_step, EINVAL. */
int griffin_draft_step(griffin_draft *draft, int32_t batch, const int32_t *prefix_len, const int32_t *n_nodes,
                       const int32_t *tokens, const int32_t *parents, const float *root_features, int32_t k,
                       int32_t *topk_tokens, float *topk_logp);

/* Extend the draft's own cache by accepted tokens: for sequence b, the
 * n_tokens[b] tokens tokens[b][0..n) (host [batch][max_tree]) at positions
 * prefix_len[b] + j, with input features features (device fp32
 * [batch][max_tree][d]; row j is the target's feature of the token before
 * token j, see griffin_read_features).  One draft pass over each chain that
 * stops once the decoder layer has written the chain's K/V to cache slots
 * prefix_len[b] + j; the caller continues with prefix_len + n_tokens.
 * Enqueued on the draft's stream, no synchronisation.  Errors: EINVAL, ETREE
 * (n_tokens outside [1, min(max_tree, max_depth + 1)]), ETOKEN, ECAPACITY,
 * EHIP. */
int griffin_draft_extend(griffin_draft *draft, int32_t batch, const int32_t *prefix_len, const int32_t *n_tokens,
                         const int32_t *tokens, const float *features);

/* Draft a tree for each of `batch` sequences by dynamic expansion (the paper
 * follows EAGLE-2's configuration: 60 draft tokens, depth 6): `depth` draft
 * passes; every expanded node proposes its top-k tokens, scored by the
 * cumulative log-probability of their path; the k best candidates of a
 * depth are expanded in the next pass; the tree is the n_total best
 * candidates of all depths (ties: the earlier candidate), numbered by depth,
 * then by rank.  root_tokens host [batch]; root_features device fp32
 * [batch][d].  Outputs, host, laid out for griffin_verify_step: n_nodes_out
 * [batch], tokens_out and parents_out [batch][max_tree], scores_out (optional)
 * [batch][max_tree] the cumulative log-probabilities (root 0).
 * Errors: EINVAL, ETREE (k, depth or n_total do not fit max_tree/max_depth),
 * and those of griffin_draft_step. */
int griffin_draft_tree(griffin_draft *draft, int32_t batch, const int32_t *prefix_len, const int32_t *root_tokens,
                       const float *root_features, int32_t k, int32_t depth, int32_t n_total,
                       int32_t *n_nodes_out, int32_t *tokens_out, int32_t *parents_out, float *scores_out);

/* Kernel classes of one verification pass, for griffin_profile_*. */
#define GRIFFIN_KC_QKV 0     /* QKV projection GEMM */
#define GRIFFIN_KC_ROPE 1    /* rotary embedding + tree K/V write */
#define GRIFFIN_KC_ATTN 2    /* prefix attention: split-KV partials */
#define GRIFFIN_KC_O 3       /* output projection GEMM */
#define GRIFFIN_KC_NORM 4    /* residual update + RMSNorm (and embedding; MoE: routing and dispatch) */
#define GRIFFIN_KC_GATE_UP 5 /* gate/up GEMM with SwiGLU (MoE: routed experts) */
#define GRIFFIN_KC_DOWN 6    /* down GEMM (MoE: routed experts) */
#define GRIFFIN_KC_LM_HEAD 7 /* LM head GEMM with per-tile argmax */
#define GRIFFIN_KC_OTHER 8   /* argmax reduction, acceptance walk */
#define GRIFFIN_KC_MERGE 9   /* split merge + ancestor (tree-key) attention */
#define GRIFFIN_KC_COUNT 10

/* Per-class timing of the launches of the classes in `class_mask` (bit k =
 * class k); 0 disables.  The GEMM classes (QKV, O, gate/up, down, LM head)
 * time themselves: each launch records, on the device wall clock, the start
 * of its earliest workgroup and the end of its latest wave (after its stores
 * complete), so the dispatch gap before the kernel is not counted (up to
 * 16384 launches between reads).  The other classes are timed with HIP
 * events recorded on the context's stream around every launch, which include
 * that gap.  Timing disables graph replay and adds work per launch, so time
 * the pass itself without it.  Errors: EINVAL, ENOMEM, EHIP. */
int griffin_profile_enable(griffin_ctx *ctx, uint32_t class_mask);

/* Wait for the stream, then return per class the summed launch durations in
 * milliseconds (ms[GRIFFIN_KC_COUNT]) and the number of launches timed
 * (launches[GRIFFIN_KC_COUNT]) since the last read or enable; resets both.
 * Errors: EINVAL, EHIP. */
int griffin_profile_read(griffin_ctx *ctx, double *ms, int64_t *launches);

#ifdef __cplusplus
}
#endif

#endif /* GRIFFIN_VERIFY_H */
