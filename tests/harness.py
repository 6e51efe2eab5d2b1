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
# MoE: a node is left out of the gates when its own or an ancestor's router has
# its last kept and first dropped expert logits closer than this (in any
# layer): the GPU router sees bf16-path activations whose relative error
# (~3e-3) moves router logits of std ~0.45 by ~1e-3, so a closer pair can
# route differently.
ROUTER_GAP = 5e-3


@dataclass
class OracleSeq:
    case: SeqCase
    logits: np.ndarray
    pred: np.ndarray
    margin: np.ndarray
    accept: "oracle.accept.AcceptResult"
    router_logits: Optional[np.ndarray]


def oracle_sequence(ow: oracle.OracleWeights, case: SeqCase) -> OracleSeq:
    res = oracle.verify_tree(ow, case.kv.fn(), case.tree, case.kv.length)
    pred = oracle.argmax_first(res.logits)
    return OracleSeq(case, res.logits, pred, oracle.top2_margin(res.logits),
                     oracle.accept_dfs(case.tree, pred), res.router_logits)


def visited_nodes(tree, pred) -> List[int]:
    """Nodes whose whole root path is accepted under predictions pred."""
    out = [0]
    for i in range(1, tree.n):
        path = tree.root_path(i)
        if all(int(tree.tokens[n]) == int(pred[int(tree.parents[n])]) for n in path):
            out.append(i)
    return out


def router_near_tie_nodes(os_: OracleSeq, top_k: int, gap: float) -> set:
    """Nodes whose own or ancestors' routing has a kept/dropped expert logit gap below `gap`."""
    if os_.router_logits is None:
        return set()
    rl = os_.router_logits                     # [L, T, E]
    srt = -np.sort(-rl, axis=-1)
    close = np.any(srt[..., top_k - 1] - srt[..., top_k] < gap, axis=0)   # [T]
    tree = os_.case.tree
    bad = set()
    for i in range(tree.n):
        if any(close[n] for n in [0] + tree.root_path(i)):
            bad.add(i)
    return bad


def check_parity(os_: OracleSeq, gpu_logits: np.ndarray, gpu_pred: np.ndarray, gpu_accept, exclude=frozenset()):
    """Assert the spec gates for one sequence; returns stats."""
    T = os_.case.tree.n
    keep = [i for i in range(T) if i not in exclude]
    ol = os_.logits[keep]
    gl = gpu_logits[keep].astype(np.float64)
    rng = ol.max(axis=1) - ol.min(axis=1)
    rel = np.abs(gl - ol).max(axis=1) / rng
    assert rel.max() <= LOGIT_REL_TOL, f"logit error {rel.max():.3e} (relative to range) above {LOGIT_REL_TOL}"
    gated = [i for i in keep if os_.margin[i] > MARGIN_GATE]
    mism = [i for i in gated if int(gpu_pred[i]) != int(os_.pred[i])]
    assert not mism, f"argmax differs at nodes {mism} (margins {[os_.margin[i] for i in mism]})"
    vis = visited_nodes(os_.case.tree, os_.pred)
    accept_gated = all(os_.margin[i] > MARGIN_GATE and i not in exclude for i in vis)
    if accept_gated:
        L, toks, _path = gpu_accept
        assert L == os_.accept.length, f"accept length {L} != oracle {os_.accept.length}"
        assert toks == os_.accept.tokens, f"accepted tokens {toks} != oracle {os_.accept.tokens}"
    return dict(max_rel=float(rel.max()), gated=len(gated), total=T, accept_checked=accept_gated,
                L=os_.accept.length)
