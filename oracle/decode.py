"""Plain causal decoding, one token at a time (fp64).

Written separately from the tree pass so that the tree pass can be pinned to
it: decoding appends each token's rotated key and value to a growing cache and
attends causally over everything cached, with no tree or mask.  The paper
calls speculative decoding lossless (Sec. 5): the tokens it emits are exactly
the target's own greedy continuation, which is what `greedy_chain` produces.
"""

from __future__ import annotations

from typing import List, Optional, Tuple

import numpy as np

from .accept import AcceptResult, argmax_first
from .model import OracleWeights, mlp, rmsnorm, rope, softmax, split_qkv


class DecodeCache:
    """Per layer: K [Hkv, n, dh] (post-rotary) and V [Hkv, n, dh], fp64."""

    def __init__(self, m, K: Optional[List[np.ndarray]] = None, V: Optional[List[np.ndarray]] = None):
        self.m = m
        if K is None:
            K = [np.zeros((m.n_kv_heads, 0, m.head_dim)) for _ in range(m.n_layers)]
            V = [np.zeros((m.n_kv_heads, 0, m.head_dim)) for _ in range(m.n_layers)]
        self.K, self.V = K, V

    def __len__(self) -> int:
        return self.K[0].shape[1]

    def copy(self) -> "DecodeCache":
        return DecodeCache(self.m, [k.copy() for k in self.K], [v.copy() for v in self.V])


def decode_step(ow: OracleWeights, cache: DecodeCache, token: int, pos: int) -> np.ndarray:
    """Logits after appending `token` at position `pos` (the cache grows by one)."""
    m = ow.shape
    Hq, Hkv, dh = m.n_q_heads, m.n_kv_heads, m.head_dim
    group = Hq // Hkv
    x = ow.embed([token])                              # [1, d]
    for l in range(m.n_layers):
        L = ow.layer(l)
        h = rmsnorm(x, L["attn_norm"], m.rms_eps)
        q, k, v = split_qkv(h, L["w_qkv"], m)
        q = rope(q[0], pos, m.rope_base)               # [Hq, dh]
        k = rope(k[0], pos, m.rope_base)               # [Hkv, dh]
        cache.K[l] = np.concatenate([cache.K[l], k[:, None, :]], axis=1)
        cache.V[l] = np.concatenate([cache.V[l], v[0][:, None, :]], axis=1)
        o = np.zeros((Hq, dh))
        for hq in range(Hq):
            hk = hq // group
            s = cache.K[l][hk] @ q[hq] / np.sqrt(dh)
            o[hq] = softmax(s) @ cache.V[l][hk]
        x = x + o.reshape(1, Hq * dh) @ L["w_o"].T
        h2 = rmsnorm(x, L["mlp_norm"], m.rms_eps)
        y, _ = mlp(h2, L, m)
        x = x + y
    return (rmsnorm(x, ow.final_norm, m.rms_eps) @ ow.lm_head().T)[0]


def prefill(ow: OracleWeights, tokens) -> DecodeCache:
    """Cache of a prompt, built by decoding it token by token from position 0."""
    cache = DecodeCache(ow.shape)
    for p, t in enumerate(tokens):
        decode_step(ow, cache, int(t), p)
    return cache


def greedy_chain(ow: OracleWeights, cache: DecodeCache, root_token: int, n: int
                 ) -> Tuple[List[int], List[float], List[np.ndarray]]:
    """The target's greedy continuation g_1..g_n after prefix + root.

    Returns the tokens, the top-2 logit margin of each prediction and the
    logits of each step (root first).  The cache is not modified."""
    from .accept import top2_margin
    c = cache.copy()
    P = len(c)
    tok, out, margins, logits_all = int(root_token), [], [], []
    for k in range(n):
        logits = decode_step(ow, c, tok, P + k)
        tok = int(argmax_first(logits))
        out.append(tok)
        margins.append(float(top2_margin(logits)))
        logits_all.append(logits)
    return out, margins, logits_all


def brute_force_accept(ow: OracleWeights, cache: DecodeCache, tree) -> AcceptResult:
    """Enumerate every root-to-leaf path, decode along it and count how many
    draft tokens agree with the target's prediction before the first miss;
    keep the longest (first leaf in id order on ties)."""
    P = len(cache)
    T = tree.n
    has_child = np.zeros(T, dtype=bool)
    for i in range(1, T):
        has_child[tree.parents[i]] = True
    best: Optional[AcceptResult] = None
    for leaf in range(T):
        if has_child[leaf]:
            continue
        path = tree.root_path(leaf)
        c = cache.copy()
        logits = decode_step(ow, c, int(tree.tokens[0]), P)
        matched: List[int] = []
        for k, node in enumerate(path):
            pred = int(argmax_first(logits))
            if int(tree.tokens[node]) != pred:
                break
            matched.append(node)
            logits = decode_step(ow, c, int(tree.tokens[node]), P + k + 1)
        res = AcceptResult(len(matched), [int(tree.tokens[n]) for n in matched]
                           + [int(argmax_first(logits))], matched)
        if best is None or res.length > best.length:
            best = res
    return best
