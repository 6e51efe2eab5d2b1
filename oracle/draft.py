"""GRIFFIN-style draft model forward and draft-tree expansion, in fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The draft model (Sec. 4.2, Fig. "Structure of GRIFFIN's draft model"): the
Token-Guided Fusion module fuses the input feature F with the embedding e of
the token, an autoregressive decoder layer follows, and the Token-Enhanced
Head splits the result into a predict feature (mapped to tokens by the
target's LM head, as in EAGLE's feature-level drafting, Sec. 3) and a regress
feature (the input feature of the next draft pass).  TGF, in the order of its
three equations in Sec. 4.2:

    h = [F, e] W_m + b_m                      (embedding fusion)
    z = [LN(h), LN(e)] W_u + b_u              (normalisation and expansion)
    o = SiLU(z) W_d + b_d + h                 (refinement, residual)

Readings (the paper gives no equations for these; listed in the design doc):
* LN is LayerNorm with its own gain and bias for h and for e (eps 1e-5);
  the expansion dimension is the appendix's 11008 (with it the 8B draft has
  the published 0.42B parameters).
* The decoder layer is one layer of the target's architecture (RMSNorm,
  rotary attention over the draft's own cache of the prefix plus the node's
  ancestors in the draft tree, SwiGLU MLP); for an MoE target its MLP is
  dense, of the experts' width.
* TEH is two linear heads with bias on the layer output y: F^P = y W_p + b_p
  and F^R = y W_r + b_r.  Logits = RMSNorm(F^P) (the target's final norm)
  times the target's LM head.
* The tree is expanded as in EAGLE-2, whose configuration the paper follows
  (App., "Draft Tree Structure": dynamic tree, 60 draft tokens, depth 6):
  every expanded node proposes its top-k tokens, scored by the cumulative
  log-probability of their path; the k best candidates of a depth are
  expanded in the next draft pass (depth passes in all); the final tree is
  the n_total best candidates of all depths (ties: the earlier candidate).
  A node's input feature is its parent's regress feature (the root's comes
  from the target).
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import Callable, List, Tuple

import numpy as np

from .model import OracleWeights, rmsnorm, rope, silu, split_qkv, mlp, to_f64
from .verify import ancestor_matrix, tree_attention


class DraftOracleWeights:
    """fp64 view of a ``workloads.gen.DraftWeights`` plus the target's shared
    embedding, final norm and LM head (from the target's OracleWeights)."""

    def __init__(self, dw, target: OracleWeights):
        self.shape = dw.shape
        self.t = {k: to_f64(v) for k, v in dw.t.items()}
        self.layer = {k: to_f64(v) for k, v in dw.layer.items()}
        self.target = target


def layernorm(x: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float) -> np.ndarray:
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def tgf(dow: DraftOracleWeights, F: np.ndarray, e: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Token-Guided Fusion of features F [T, d] and token embeddings e [T, d]:
    returns (h, o)."""
    t, eps = dow.t, dow.shape.ln_eps
    h = np.concatenate([F, e], axis=1) @ t["w_m"].T + t["b_m"]
    z = np.concatenate([layernorm(h, t["ln_h_g"], t["ln_h_b"], eps),
                        layernorm(e, t["ln_x_g"], t["ln_x_b"], eps)], axis=1) @ t["w_u"].T + t["b_u"]
    o = silu(z) @ t["w_d"].T + t["b_d"] + h
    return h, o


@dataclass
class DraftResult:
    logits: np.ndarray    # [T, V]
    predict: np.ndarray   # F^P [T, d]
    regress: np.ndarray   # F^R [T, d]
    h: np.ndarray         # TGF fusion [T, d]
    o: np.ndarray         # TGF output = decoder-layer input [T, d]
    y: np.ndarray         # decoder-layer output [T, d]
    k: np.ndarray = None  # the decoder layer's K of the nodes [T, Hkv, dh], post-rotary
    v: np.ndarray = None  # and V [T, Hkv, dh]: what the pass adds to the draft's cache


def draft_forward(dow: DraftOracleWeights, tree, feats_in: np.ndarray, prefix_kv: Tuple[np.ndarray, np.ndarray],
                  prefix_len: int) -> DraftResult:
    """One draft pass over the nodes of `tree` (node 0 the root, at position
    prefix_len + depth): feats_in [T, d] input features, prefix_kv the draft
    layer's cached prefix (K post-rotary, V; [Hkv, P, dh] each)."""
    m = dow.shape.target
    T, P = tree.n, prefix_len
    Hq, dh = m.n_q_heads, m.head_dim
    pos = P + tree.depths()
    visible = np.concatenate([np.ones((T, P), dtype=bool), ancestor_matrix(tree.parents)], axis=1)
    e = dow.target.embed(tree.tokens)
    h, o = tgf(dow, np.asarray(feats_in, dtype=np.float64), e)
    L = dow.layer
    x = o
    a = rmsnorm(x, L["attn_norm"], m.rms_eps)
    q, k, v = split_qkv(a, L["w_qkv"], m)
    q = rope(q, pos[:, None], m.rope_base)
    k = rope(k, pos[:, None], m.rope_base)
    att = tree_attention(q, k, v, prefix_kv[0], prefix_kv[1], visible)
    x = x + att.reshape(T, Hq * dh) @ L["w_o"].T
    y2, _ = mlp(rmsnorm(x, L["mlp_norm"], m.rms_eps), L, dow.shape.layer)
    y = x + y2
    t = dow.t
    fp = y @ t["w_p"].T + t["b_p"]
    fr = y @ t["w_r"].T + t["b_r"]
    logits = rmsnorm(fp, dow.target.final_norm, m.rms_eps) @ dow.target.lm_head().T
    return DraftResult(logits, fp, fr, h, o, y, k, v)


def topk_logprobs(logits: np.ndarray, k: int) -> Tuple[np.ndarray, np.ndarray]:
    """Per row: the k most probable tokens (ties: lower id) and their
    log-probabilities under softmax(logits)."""
    lg = np.asarray(logits, dtype=np.float64)
    mx = lg.max(axis=-1, keepdims=True)
    lse = mx + np.log(np.exp(lg - mx).sum(axis=-1, keepdims=True))
    logp = lg - lse
    order = np.argsort(-lg, axis=-1, kind="stable")[:, :k]
    return order.astype(np.int32), np.take_along_axis(logp, order, axis=-1)


@dataclass
class Expansion:
    tree: object                 # the drafted tree (workloads.gen.Tree), BFS by depth
    scores: np.ndarray           # cumulative log-probability of every tree node (root 0)
    passes: List[object]         # the tree of every draft pass (root + expanded nodes so far)
    candidate_scores: np.ndarray  # score of every candidate, in generation order


StepFn = Callable[[object, np.ndarray], Tuple[np.ndarray, np.ndarray, np.ndarray]]


def expand_tree(root_token: int, root_feature: np.ndarray, step: StepFn, k: int, depth: int,
                n_total: int, tree_cls) -> Expansion:
    """EAGLE-2-style dynamic expansion (reading in the module docstring).

    step(pass_tree, feats_in) runs one draft pass over the expanded nodes and
    returns per node (top-k tokens [T, k], their log-probabilities [T, k],
    regress features [T, d]); only the rows expanded in this pass are used.
    tree_cls(tokens, parents) builds a tree."""
    p_tok, p_par, p_cand, p_score = [int(root_token)], [-1], [-1], [0.0]
    feats = [np.asarray(root_feature, dtype=np.float64)]
    cands: List[Tuple[int, int, int, float]] = []   # (depth, expanded parent node, token, score)
    frontier, passes = [0], []
    for t in range(depth):
        ptree = tree_cls(np.array(p_tok, dtype=np.int32), np.array(p_par, dtype=np.int32))
        passes.append(ptree)
        tok, logp, regress = step(ptree, np.stack(feats))
        new = []
        for r in frontier:
            for j in range(k):
                cands.append((t + 1, r, int(tok[r, j]), p_score[r] + float(logp[r, j])))
                new.append(len(cands) - 1)
        if t + 1 == depth:
            break
        best = sorted(new, key=lambda c: (-cands[c][3], c))[:k]
        frontier = []
        for c in best:
            _, r, token, score = cands[c]
            p_tok.append(token)
            p_par.append(r)
            p_cand.append(c)
            p_score.append(score)
            feats.append(np.asarray(regress[r], dtype=np.float64))
            frontier.append(len(p_tok) - 1)
    chosen = sorted(range(len(cands)), key=lambda c: (-cands[c][3], c))[:n_total]
    rank = {c: i for i, c in enumerate(chosen)}
    order = sorted(chosen, key=lambda c: (cands[c][0], rank[c]))
    index = {c: i + 1 for i, c in enumerate(order)}
    tokens = [int(root_token)] + [cands[c][2] for c in order]
    parents = [-1]
    for c in order:
        pc = p_cand[cands[c][1]]   # candidate that the expanded parent node came from (-1: the root)
        parents.append(0 if pc < 0 else index[pc])
    scores = np.array([0.0] + [cands[c][3] for c in order])
    return Expansion(tree_cls(np.array(tokens, dtype=np.int32), np.array(parents, dtype=np.int32)), scores,
                     passes, np.array([c[3] for c in cands]))
