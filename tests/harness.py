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
            kv = prefix_kv_synthetic(m, seq, w.prefix_len, w.weight_seed)
    tree, path = gen.workload_tree(w, tree_index, seq)
    greedy, margins = [], []
    if path:
        greedy, margins, _ = oracle.greedy_chain(ow, kv.decode_cache(m), int(tree.tokens[0]), len(path))
        tree = gen.apply_plant(tree, path, greedy)
    return SeqCase(toks, kv, tree, path, greedy, margins)
