"""One tree-verification pass of the target model (fp64).

The paper (Sec. 3) has the target verify all draft tokens of a cycle in a
single forward pass, and (Sec. 4.1) the draft tokens of one cycle form a tree
because several top-k candidates are kept per position.  A node therefore sees
the prefix plus exactly its own root path: for node i the keys are the cached
prefix positions 0..P-1 and the tree nodes j that are ancestors of i or i
itself.  Node i sits at sequence position P + depth(i), so its logits are the
ones plain causal decoding would produce after prefix + root path.

Readings where the paper is silent (listed with the rest in the design notes):
the root (node 0) is the last accepted token, not yet in the cache, at
position P; rotation uses the node's depth-derived position; the prefix cache
holds post-rotary keys.
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import Callable, List, Optional, Tuple

import numpy as np

from .model import OracleWeights, mlp, rmsnorm, rope, softmax, split_qkv


@dataclass
class VerifyResult:
    logits: np.ndarray                      # [T, V]
    hidden: np.ndarray                      # [T, d] residual stream before the final norm
    tree_k: List[np.ndarray]                # per layer [T, Hkv, dh], post-rotary
    tree_v: List[np.ndarray]                # per layer [T, Hkv, dh]
    router_logits: Optional[np.ndarray]     # [L, T, E] for MoE targets


def ancestor_matrix(parents: np.ndarray) -> np.ndarray:
    """vis[i, j] = True iff node j lies on the path from the root to node i."""
    T = len(parents)
    vis = np.zeros((T, T), dtype=bool)
    for i in range(T):
        j = i
        while j >= 0:
            vis[i, j] = True
            j = int(parents[j]) if j > 0 else -1
    return vis


def tree_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, Kp: np.ndarray, Vp: np.ndarray,
                   visible: np.ndarray) -> np.ndarray:
    """Masked attention of the tree nodes.

    q [T, Hq, dh]; k, v [T, Hkv, dh] (the nodes' own keys and values, sequence
    slots P..P+T-1); Kp, Vp [Hkv, P, dh] (the cached prefix); visible [T, P+T]
    says which keys each node may see.  Query head h reads KV head
    h // (Hq / Hkv).  Returns o [T, Hq, dh]."""
    T, Hq, dh = q.shape
    group = Hq // k.shape[1]
    o = np.zeros((T, Hq, dh))
    for hq in range(Hq):
        hk = hq // group
        keys = np.concatenate([Kp[hk], k[:, hk, :]], axis=0)            # [P + T, dh]
        vals = np.concatenate([Vp[hk], v[:, hk, :]], axis=0)
        s = (q[:, hq, :] @ keys.T) / np.sqrt(dh)                         # [T, P + T]
        s = np.where(visible, s, -np.inf)
        o[:, hq, :] = softmax(s, axis=-1) @ vals
    return o


def verify_tree(ow: OracleWeights, prefix_kv: Callable[[int], Tuple[np.ndarray, np.ndarray]],
                tree, prefix_len: int) -> VerifyResult:
    """Logits of every tree node.

    prefix_kv(l) returns the cached prefix of layer l as fp64 (K [Hkv, P, dh]
    post-rotary, V [Hkv, P, dh])."""
    m = ow.shape
    T, P = tree.n, prefix_len
    Hq, Hkv, dh = m.n_q_heads, m.n_kv_heads, m.head_dim
    pos = P + tree.depths()
    vis = ancestor_matrix(tree.parents)
    visible = np.concatenate([np.ones((T, P), dtype=bool), vis], axis=1)   # [T, P + T]

    x = ow.embed(tree.tokens)
    tree_k, tree_v, routers = [], [], []
    for l in range(m.n_layers):
        L = ow.layer(l)
        h = rmsnorm(x, L["attn_norm"], m.rms_eps)
        q, k, v = split_qkv(h, L["w_qkv"], m)
        q = rope(q, pos[:, None], m.rope_base)
        k = rope(k, pos[:, None], m.rope_base)
        tree_k.append(k)
        tree_v.append(v)
        Kp, Vp = prefix_kv(l)
        o = tree_attention(q, k, v, Kp, Vp, visible)
        x = x + o.reshape(T, Hq * dh) @ L["w_o"].T
        h2 = rmsnorm(x, L["mlp_norm"], m.rms_eps)
        y, rl = mlp(h2, L, m)
        if rl is not None:
            routers.append(rl)
        x = x + y
    logits = rmsnorm(x, ow.final_norm, m.rms_eps) @ ow.lm_head().T
    return VerifyResult(logits, x, tree_k, tree_v, np.stack(routers) if routers else None)
