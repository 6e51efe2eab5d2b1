"""Shared test harness: builds oracle-side inputs from the seeded workloads.

Only tests import this module.  It may use the oracle (the tests are the
oracle's users); it never feeds anything produced by the HIP library back into
the oracle.
"""

from __future__ import annotations

from dataclasses import dataclass, replace
from typing import Dict, List, Optional, Tuple

import numpy as np
import torch

from workloads import gen
from workloads.configs import ModelShape, Workload, get_workload

import oracle
from oracle.decode import DecodeCache


def micro_shape(**kw) -> ModelShape:
    base = dict(name="micro", n_layers=2, d_model=64, n_q_heads=4, n_kv_heads=2, head_dim=16,
                d_ff=96, vocab=97, rms_eps=1e-5, rope_base=10000.0)
    base.update(kw)
    return ModelShape(**base)


def bf16_round(a: np.ndarray) -> np.ndarray:
    """fp64 -> nearest bf16 (RNE) -> fp64."""
    return torch.from_numpy(np.ascontiguousarray(a)).to(torch.bfloat16).to(torch.float64).numpy()


@dataclass
class PrefixKV:
    """Cached prefix of one sequence as the verify pass receives it: bf16
    values (here upcast to fp64), K post-rotary.  K, V: per layer [Hkv, P, dh]."""
    K: List[np.ndarray]
    V: List[np.ndarray]

    @property
    def length(self) -> int:
        return self.K[0].shape[1]

    def fn(self):
        return lambda l: (self.K[l], self.V[l])

    def decode_cache(self, m) -> DecodeCache:
        return DecodeCache(m, [k.copy() for k in self.K], [v.copy() for v in self.V])


def prefix_kv_prefill(ow: oracle.OracleWeights, tokens) -> PrefixKV:
    """fp64 oracle prefill of the prefix tokens, rounded to bf16."""
    c = oracle.prefill(ow, tokens)
    return PrefixKV([bf16_round(k) for k in c.K], [bf16_round(v) for v in c.V])


def prefix_kv_synthetic(m: ModelShape, seq: int, P: int, seed: int = 0) -> PrefixKV:
    Ks, Vs = [], []
    for l in range(m.n_layers):
        k, v = gen.synthetic_kv(m, l, seq, P, seed)
        Ks.append(k.to(torch.float64).numpy())
        Vs.append(v.to(torch.float64).numpy())
    return PrefixKV(Ks, Vs)


@dataclass
class SeqCase:
    prefix_tokens: np.ndarray
    kv: PrefixKV
    tree: gen.Tree
    plant_path: List[int]
    greedy: List[int]          # oracle greedy continuation after prefix + root (len = plant length)
    greedy_margins: List[float]


def build_sequence(ow: oracle.OracleWeights, w: Workload, tree_index: int, seq: int = 0,
                   kv: Optional[PrefixKV] = None) -> SeqCase:
    """One sequence of a workload: prefix KV, tree, and the planted greedy path
    (computed by the oracle's own causal decoding)."""
    m = w.model
    toks = gen.prefix_tokens(w, seq)
    if kv is None:
        if w.kv_source == "prefill":
            kv = prefix_kv_prefill(ow, toks)
        else:
            kv = prefix_kv_synthetic(m, seq, w.prefix_of(seq), w.weight_seed)
    tree, path = gen.workload_tree(w, tree_index, seq)
    greedy, margins = [], []
    if path:
        greedy, margins, _ = oracle.greedy_chain(ow, kv.decode_cache(m), int(tree.tokens[0]), len(path))
        tree = gen.apply_plant(tree, path, greedy)
    return SeqCase(toks, kv, tree, path, greedy, margins)


# ------------------------------------------------------------ GPU parity ----

LOGIT_REL_TOL = 2e-2      # max |gpu - oracle| per row, relative to the oracle row's range
MARGIN_GATE = 1e-2        # argmax / acceptance compared bit-exactly where the top-2 margin exceeds this
# A tighter bound on the same statistic, so that a numerical regression far
# below the acceptance gate is still caught: the measured error is 3e-6 (tiny)
# to 8e-5 (Mixtral shape, 32 layers) of the row range.
REGRESS_REL_TOL = 1e-3
# MoE: the device's router logits are read back, so the gates know exactly
# where the GPU chose other experts than the oracle.  Every such choice must
# be a near tie (the oracle's kept/dropped gap within twice the largest
# router-logit error measured on the same pass, never below ROUTER_GAP_MIN);
# the nodes below it are left out of the gates (their inputs legitimately
# differ) and counted.
ROUTER_GAP_MIN = 1e-4


def router_check(os_: "OracleSeq", gpu_rl: np.ndarray, top_k: int):
    """Compare the device's routing with the oracle's for one sequence.

    gpu_rl [L, T, E]: the device's router logits.  A node's routing at layer
    l depends on its ancestors only through their keys and values at layer l,
    which precede the ancestors' own routing at that layer; so a node's
    router logits are compared up to and including the first layer at which
    it or an ancestor chose other experts than the oracle (after that its
    inputs legitimately differ).  Asserts that every such choice is a near
    tie.  Returns (measured error, gap, nodes with a differing choice on
    their root path, nodes with an oracle gap below `gap` on their root path)."""
    orl = os_.router_logits
    L, T, E = orl.shape
    tree = os_.case.tree
    o_top = np.sort(np.argsort(-orl, axis=-1, kind="stable")[..., :top_k], axis=-1)
    g_top = np.sort(np.argsort(-gpu_rl[:, :T].astype(np.float64), axis=-1, kind="stable")[..., :top_k], axis=-1)
    flip = np.any(o_top != g_top, axis=-1)                                   # [L, T]
    first = np.where(flip.any(axis=0), flip.argmax(axis=0), L)              # first differing layer per node
    srt = -np.sort(-orl, axis=-1)
    gaps = srt[..., top_k - 1] - srt[..., top_k]                             # [L, T]
    anc = [[0] + tree.root_path(i) for i in range(T)]
    last = [min(int(first[n]) for n in anc[i]) for i in range(T)]            # first divergence on the root path
    err = 0.0
    for i in range(T):
        upto = min(L - 1, last[i])
        err = max(err, float(np.abs(gpu_rl[: upto + 1, i] - orl[: upto + 1, i]).max()))
    gap = max(ROUTER_GAP_MIN, 2.0 * err)
    for i in range(T):
        if first[i] < L and first[i] <= last[i]:
            l = int(first[i])
            assert gaps[l, i] <= gap, f"node {i} layer {l}: experts differ at an oracle gap {gaps[l, i]:.2e} > {gap:.2e}"
    diverged = {i for i in range(T) if last[i] < L}
    near = {i for i in range(T) if any(np.any(gaps[:, n] < gap) for n in anc[i])}
    return err, gap, diverged, near


@dataclass
class OracleSeq:
    case: SeqCase
    logits: np.ndarray
    pred: np.ndarray
    margin: np.ndarray
    accept: "oracle.accept.AcceptResult"
    router_logits: Optional[np.ndarray]
    hidden: np.ndarray          # [T, d] residual stream after the last layer


def oracle_sequence(ow: oracle.OracleWeights, case: SeqCase) -> OracleSeq:
    res = oracle.verify_tree(ow, case.kv.fn(), case.tree, case.kv.length)
    pred = oracle.argmax_first(res.logits)
    return OracleSeq(case, res.logits, pred, oracle.top2_margin(res.logits),
                     oracle.accept_dfs(case.tree, pred), res.router_logits, res.hidden)


def visited_nodes(tree, pred) -> List[int]:
    """Nodes whose whole root path is accepted under predictions pred."""
    out = [0]
    for i in range(1, tree.n):
        path = tree.root_path(i)
        if all(int(tree.tokens[n]) == int(pred[int(tree.parents[n])]) for n in path):
            out.append(i)
    return out


def check_parity(os_: OracleSeq, gpu_logits: np.ndarray, gpu_pred: np.ndarray, gpu_accept, exclude=frozenset(),
                 regress_tol: float = REGRESS_REL_TOL):
    """Assert the spec gates for one sequence; returns stats.

    * logits: per row max |gpu - oracle| <= LOGIT_REL_TOL of the oracle row's
      range (and <= regress_tol, the regression bound);
    * argmax bit-exact at every node whose oracle top-2 margin exceeds
      MARGIN_GATE; elsewhere the GPU's token must be one whose oracle logit is
      within MARGIN_GATE of the row's maximum (a valid greedy choice up to
      rounding);
    * acceptance: the GPU's walk must be exactly the DFS walk over its own
      predictions (always checked), and equal to the oracle's result when every
      node the oracle's walk visits clears the margin gate."""
    T = os_.case.tree.n
    keep = [i for i in range(T) if i not in exclude]
    ol = os_.logits[keep]
    gl = gpu_logits[keep].astype(np.float64)
    rng = ol.max(axis=1) - ol.min(axis=1)
    rel = np.abs(gl - ol).max(axis=1) / rng
    assert rel.max() <= LOGIT_REL_TOL, f"logit error {rel.max():.3e} (relative to range) above {LOGIT_REL_TOL}"
    assert rel.max() <= regress_tol, f"logit error {rel.max():.3e} above the regression bound {regress_tol}"
    gated = [i for i in keep if os_.margin[i] > MARGIN_GATE]
    mism = [i for i in gated if int(gpu_pred[i]) != int(os_.pred[i])]
    assert not mism, f"argmax differs at nodes {mism} (margins {[os_.margin[i] for i in mism]})"
    for i in keep:
        if i not in gated:
            row = os_.logits[i]
            assert row[int(gpu_pred[i])] >= row.max() - MARGIN_GATE, f"node {i}: token {gpu_pred[i]} is no near-tie"
    L, toks, path = gpu_accept
    own = oracle.accept_dfs(os_.case.tree, np.asarray(gpu_pred[:T]))
    assert (L, list(toks), list(path)) == (own.length, list(own.tokens), list(own.path)), \
        f"walk {(L, toks, path)} != DFS over the GPU's own predictions {own}"
    vis = visited_nodes(os_.case.tree, os_.pred)
    accept_gated = all(os_.margin[i] > MARGIN_GATE and i not in exclude for i in vis)
    if accept_gated:
        assert L == os_.accept.length, f"accept length {L} != oracle {os_.accept.length}"
        assert toks == os_.accept.tokens, f"accepted tokens {toks} != oracle {os_.accept.tokens}"
    return dict(max_rel=float(rel.max()), gated=len(gated), total=T, accept_checked=accept_gated,
                L=os_.accept.length)
