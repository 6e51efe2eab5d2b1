"""Seeded generators for weights, prefix tokens, prefix KV and draft trees.

Weights and synthetic KV values come from a counter-based generator so that
any element can be produced on any device, in any order, with identical bits:

* hash: the 32-bit "lowbias32" integer mixer (C. Wellons, "Prospecting for
  Hash Functions", 2018): x ^= x>>16; x *= 0x7feb352d; x ^= x>>15;
  x *= 0x846ca68b; x ^= x>>16, all modulo 2^32.
* element value: the four bytes of hash(index) are summed (an Irwin-Hall sum
  of four discrete uniforms on 0..255), centred, scaled by std/147.8006 in
  fp32 (one correctly rounded IEEE multiply) and rounded to bf16 (RNE).

Only integer arithmetic, one fp32 multiply and one bf16 rounding are involved,
so torch on the CPU and torch on the GPU give the same bits; a GPU test checks
that.  The values are bounded by about 3.45 std and have the requested std.

Trees and prefix tokens are drawn with numpy's PCG64 on the host.
"""

from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from .configs import ModelShape, Workload

MASK32 = 0xFFFFFFFF
# std of the sum of four independent uniforms on {0..255}: sqrt(4*(256^2-1)/12)
_IH4_STD = math.sqrt(4.0 * (256.0 * 256.0 - 1.0) / 12.0)
_CHUNK = 1 << 25


def _mul32(x: torch.Tensor, c: int) -> torch.Tensor:
    """(x * c) mod 2^32 for int64 tensors holding values in [0, 2^32)."""
    lo = c & 0xFFFF
    hi = c >> 16
    return (x * lo + (((x * hi) & 0xFFFF) << 16)) & MASK32


def mix32(x: torch.Tensor) -> torch.Tensor:
    x = x ^ (x >> 16)
    x = _mul32(x, 0x7FEB352D)
    x = x ^ (x >> 15)
    x = _mul32(x, 0x846CA68B)
    x = x ^ (x >> 16)
    return x


def _mix32_int(x: int) -> int:
    x &= MASK32
    x ^= x >> 16
    x = (x * 0x7FEB352D) & MASK32
    x ^= x >> 15
    x = (x * 0x846CA68B) & MASK32
    x ^= x >> 16
    return x


def stream_keys(seed: int, stream: int) -> tuple[int, int]:
    k1 = _mix32_int((seed & MASK32) ^ 0x2545F491)
    k2 = _mix32_int(k1 ^ (stream & MASK32))
    return k1, k2


def hashed_normal_bf16(numel: int, seed: int, stream: int, std: float,
                       device: torch.device | str = "cpu", start: int = 0) -> torch.Tensor:
    """Elements start..start+numel-1 of stream `stream` as a flat bf16 tensor."""
    device = torch.device(device)
    assert start + numel <= (1 << 32), "stream index space is 32-bit"
    k1, k2 = stream_keys(seed, stream)
    scale = torch.tensor(std / _IH4_STD, dtype=torch.float32, device=device)
    out = torch.empty(numel, dtype=torch.bfloat16, device=device)
    for c0 in range(0, numel, _CHUNK):
        c1 = min(numel, c0 + _CHUNK)
        idx = torch.arange(start + c0, start + c1, dtype=torch.int64, device=device)
        h = mix32(idx ^ k2)
        h = mix32((h + k1) & MASK32)
        s = (h & 255) + ((h >> 8) & 255) + ((h >> 16) & 255) + (h >> 24) - 510
        out[c0:c1] = (s.to(torch.float32) * scale).to(torch.bfloat16)
        del idx, h, s
    return out


# ---------------------------------------------------------------- weights ----

# stream ids
_S_EMBED, _S_LMHEAD = 1, 3
_S_LAYER_BASE, _S_LAYER_STRIDE = 1000, 16
_S_QKV, _S_O, _S_GU, _S_DOWN, _S_ROUTER, _S_ATTN_NORM, _S_MLP_NORM = 0, 1, 2, 3, 4, 5, 6
_S_FINAL_NORM = 5
_S_KV_BASE = 1 << 20


def _layer_stream(layer: int, which: int) -> int:
    return _S_LAYER_BASE + layer * _S_LAYER_STRIDE + which


@dataclass
class ModelWeights:
    """bf16 tensors in the layouts the verify library takes.

    embed      [V, d]
    lm_head    [V, d]
    final_norm [d]
    per layer:
      attn_norm, mlp_norm  [d]
      w_qkv      [(Hq + 2 Hkv) * dh, d]   rows: all q heads, then k heads, then v heads
      w_o        [d, Hq * dh]
      w_gate_up  dense [2F, d] (gate rows then up rows); MoE [E, 2F, d]
      w_down     dense [d, F];                            MoE [E, d, F]
      w_router   MoE [E, d]; None for dense
    """
    shape: ModelShape
    embed: torch.Tensor
    lm_head: torch.Tensor
    final_norm: torch.Tensor
    layers: List[Dict[str, Optional[torch.Tensor]]]

    def to(self, device) -> "ModelWeights":
        mv = lambda t: None if t is None else t.to(device)  # noqa: E731
        return ModelWeights(self.shape, mv(self.embed), mv(self.lm_head), mv(self.final_norm),
                            [{k: mv(v) for k, v in L.items()} for L in self.layers])

    def nbytes(self) -> int:
        n = self.embed.numel() + self.lm_head.numel() + self.final_norm.numel()
        for L in self.layers:
            n += sum(v.numel() for v in L.values() if v is not None)
        return 2 * n


def norm_gain(d: int, seed: int, stream: int, gain_std: float, device="cpu") -> torch.Tensor:
    """RMSNorm gain [d]: bf16(1 + N(0, gain_std^2)) from its own stream, so a
    dropped, swapped or mis-indexed gain changes the result."""
    v = hashed_normal_bf16(d, seed, stream, gain_std, device).float()
    return (v + 1.0).to(torch.bfloat16)


def make_weights(m: ModelShape, seed: int = 0, device="cpu") -> ModelWeights:
    d, f, E = m.d_model, m.d_ff, m.n_experts
    std = m.weight_std

    def mat(stream: int, *shape: int) -> torch.Tensor:
        n = int(np.prod(shape))
        return hashed_normal_bf16(n, seed, stream, std, device).view(*shape)

    layers = []
    for l in range(m.n_layers):
        L: Dict[str, Optional[torch.Tensor]] = {
            "attn_norm": norm_gain(d, seed, _layer_stream(l, _S_ATTN_NORM), m.gain_std, device),
            "mlp_norm": norm_gain(d, seed, _layer_stream(l, _S_MLP_NORM), m.gain_std, device),
            "w_qkv": mat(_layer_stream(l, _S_QKV), m.qkv_rows, d),
            "w_o": mat(_layer_stream(l, _S_O), d, m.n_q_heads * m.head_dim),
        }
        if E == 1:
            L["w_gate_up"] = mat(_layer_stream(l, _S_GU), 2 * f, d)
            L["w_down"] = mat(_layer_stream(l, _S_DOWN), d, f)
            L["w_router"] = None
        else:
            L["w_gate_up"] = mat(_layer_stream(l, _S_GU), E, 2 * f, d)
            L["w_down"] = mat(_layer_stream(l, _S_DOWN), E, d, f)
            L["w_router"] = mat(_layer_stream(l, _S_ROUTER), E, d)
        layers.append(L)
    return ModelWeights(m, mat(_S_EMBED, m.vocab, d), mat(_S_LMHEAD, m.vocab, d),
                        norm_gain(d, seed, _S_FINAL_NORM, m.gain_std, device), layers)


# ------------------------------------------------------------ draft model ----

_S_DRAFT_BASE = 500   # TGF / TEH tensors: _S_DRAFT_BASE + index below
_S_DRAFT_LAYER = 600  # the draft's decoder layer (qkv, o, gate/up, down)
_DRAFT_TENSORS = ("w_m", "b_m", "ln_h_g", "ln_h_b", "ln_x_g", "ln_x_b", "w_u", "b_u", "w_d", "b_d",
                  "w_p", "b_p", "w_r", "b_r")


@dataclass
class DraftWeights:
    """bf16 tensors of a draft model (matrices [out, in] like the target's):

    w_m [d, 2d], b_m [d]            fusion of [feature, token embedding]
    ln_h_g, ln_h_b, ln_x_g, ln_x_b  LayerNorm gains and biases [d]
    w_u [e, 2d], b_u [e]            up projection of [LN(h), LN(embedding)]
    w_d [d, e], b_d [d]             down projection
    layer                           one decoder layer, keys as ModelWeights.layers[l]
    w_p, w_r [d, d], b_p, b_r [d]   the two heads (predict, regress)
    The embedding, final norm and LM head are the target's."""
    shape: "DraftShape"
    t: Dict[str, torch.Tensor]
    layer: Dict[str, Optional[torch.Tensor]]

    def to(self, device) -> "DraftWeights":
        return DraftWeights(self.shape, {k: v.to(device) for k, v in self.t.items()},
                            {k: None if v is None else v.to(device) for k, v in self.layer.items()})


def make_draft_weights(ds, seed: int = 7, device="cpu") -> DraftWeights:
    """Random-init draft weights: matrices and biases N(0, std^2) with the
    target's std; LayerNorm gains 1 + N(0, 0.1^2) and biases N(0, 0.1^2); the
    decoder layer's RMSNorm gains 1 + N(0, gain_std^2) like the target's."""
    m, d, e = ds.target, ds.target.d_model, ds.tgf_dim
    std = m.weight_std
    shapes = {"w_m": (d, 2 * d), "b_m": (d,), "ln_h_g": (d,), "ln_h_b": (d,), "ln_x_g": (d,), "ln_x_b": (d,),
              "w_u": (e, 2 * d), "b_u": (e,), "w_d": (d, e), "b_d": (d,), "w_p": (d, d), "b_p": (d,),
              "w_r": (d, d), "b_r": (d,)}
    t = {}
    for i, name in enumerate(_DRAFT_TENSORS):
        shp = shapes[name]
        n = int(np.prod(shp))
        if name.startswith("ln_"):
            v = hashed_normal_bf16(n, seed, _S_DRAFT_BASE + i, 0.1, device).float()
            t[name] = (v + 1.0 if name.endswith("_g") else v).to(torch.bfloat16).view(*shp)
        else:
            t[name] = hashed_normal_bf16(n, seed, _S_DRAFT_BASE + i, std, device).view(*shp)
    def mat(which: int, *shape: int) -> torch.Tensor:
        return hashed_normal_bf16(int(np.prod(shape)), seed, _S_DRAFT_LAYER + which, std, device).view(*shape)

    layer = {"attn_norm": norm_gain(d, seed, _S_DRAFT_LAYER + 4, m.gain_std, device),
             "mlp_norm": norm_gain(d, seed, _S_DRAFT_LAYER + 5, m.gain_std, device),
             "w_qkv": mat(0, m.qkv_rows, d),
             "w_o": mat(1, d, m.n_q_heads * m.head_dim), "w_gate_up": mat(2, 2 * m.d_ff, d),
             "w_down": mat(3, d, m.d_ff), "w_router": None}
    return DraftWeights(ds, t, layer)


def draft_root_features(d: int, batch: int, seed: int = 11, device="cpu") -> torch.Tensor:
    """Stand-in for the target's last hidden state at each sequence's root:
    fp32 [batch, d], entries N(0, 1) rounded to bf16 (the same bits on both sides)."""
    return hashed_normal_bf16(batch * d, seed, 0, 1.0, device).float().view(batch, d)


# ------------------------------------------------------------------ prefix ----

def prefix_tokens(w: Workload, seq: int = 0) -> np.ndarray:
    rng = np.random.default_rng(w.prefix_seed + 7919 * seq)
    return rng.integers(0, w.model.vocab, size=w.prefix_of(seq), dtype=np.int64).astype(np.int32)


def kv_std(m: ModelShape) -> float:
    """Scale of a random-init model's K and V entries: unit-RMS input times
    d_model weights of std `weight_std`."""
    return m.weight_std * math.sqrt(m.d_model)


def synthetic_kv(m: ModelShape, layer: int, seq: int, prefix_len: int, seed: int = 0,
                 device="cpu") -> tuple[torch.Tensor, torch.Tensor]:
    """Prefix K (post-rotary) and V of one (layer, sequence): bf16 [Hkv, P, dh] each."""
    n = m.n_kv_heads * prefix_len * m.head_dim
    base = _S_KV_BASE + 2 * (layer * 4096 + seq)
    k = hashed_normal_bf16(n, seed, base, kv_std(m), device)
    v = hashed_normal_bf16(n, seed, base + 1, kv_std(m), device)
    shp = (m.n_kv_heads, prefix_len, m.head_dim)
    return k.view(shp), v.view(shp)


# ------------------------------------------------------------------- trees ----

@dataclass
class Tree:
    """Draft tree; node 0 is the root (the last accepted token, not yet cached).

    Nodes are numbered breadth-first by depth, so parents[i] < i for i >= 1."""
    tokens: np.ndarray   # int32 [T]
    parents: np.ndarray  # int32 [T]; parents[0] = -1

    @property
    def n(self) -> int:
        return int(self.tokens.shape[0])

    def depths(self) -> np.ndarray:
        d = np.zeros(self.n, dtype=np.int32)
        for i in range(1, self.n):
            d[i] = d[self.parents[i]] + 1
        return d

    def root_path(self, i: int) -> List[int]:
        """Node ids from depth 1 down to node i (root excluded)."""
        path = []
        while i > 0:
            path.append(i)
            i = int(self.parents[i])
        return path[::-1]

    def copy(self) -> "Tree":
        return Tree(self.tokens.copy(), self.parents.copy())


def tree_seed(w: Workload, index: int, seq: int = 0) -> int:
    return w.tree_seed + index + 100003 * seq


def random_tree(widths: Sequence[int], vocab: int, seed: int) -> tuple[Tree, np.random.Generator]:
    """Each depth-k node picks its parent uniformly among the depth-(k-1) nodes."""
    rng = np.random.default_rng(seed)
    T = 1 + int(sum(widths))
    tokens = np.zeros(T, dtype=np.int32)
    parents = np.full(T, -1, dtype=np.int32)
    tokens[0] = rng.integers(0, vocab)
    prev = [0]
    nxt = 1
    for width in widths:
        cur = []
        for _ in range(width):
            parents[nxt] = prev[int(rng.integers(0, len(prev)))]
            tokens[nxt] = rng.integers(0, vocab)
            cur.append(nxt)
            nxt += 1
        prev = cur
    return Tree(tokens, parents), rng


@dataclass
class SampledCase:
    """Inputs of the stochastic (temperature > 0) acceptance for one tree."""
    tree: Tree
    logits: np.ndarray    # float32 [T, V] target logits at every node
    q: Optional[np.ndarray]  # float32 [T, V] draft distribution of each node's children (None: deterministic)
    u_accept: np.ndarray  # float32 [T] uniform for the test at each child
    u_final: np.ndarray   # float32 [T] uniform for the token drawn at each node


def sampled_case(widths: Sequence[int], vocab: int, seed: int, temperature: float = 1.0,
                 logit_std: float = 2.0, draft_noise: float = 1.0) -> SampledCase:
    """A synthetic draft tree with the inputs the stochastic acceptance reads.

    Target logits are i.i.d. N(0, logit_std^2).  The draft at node u is
    proportional to exp(logits_u / temperature + N(0, draft_noise^2)), a
    drafter correlated with the target.  Every node's children take tokens
    drawn from its draft distribution without replacement (numpy's
    generator), as a sampling drafter would; the shape is `random_tree`'s."""
    shape, rng = random_tree(widths, vocab, seed)
    T = shape.n
    logits = rng.normal(0.0, logit_std, size=(T, vocab))
    z = logits / temperature + rng.normal(0.0, draft_noise, size=(T, vocab))
    q = np.exp(z - z.max(axis=1, keepdims=True))
    q /= q.sum(axis=1, keepdims=True)
    tokens = np.zeros(T, dtype=np.int32)
    tokens[0] = rng.integers(0, vocab)
    for u in range(T):
        kids = [c for c in range(1, T) if shape.parents[c] == u]
        if kids:
            draws = rng.choice(vocab, size=len(kids), replace=False, p=q[u])
            for c, t in zip(kids, draws):
                tokens[c] = int(t)
    return SampledCase(Tree(tokens, shape.parents.copy()), logits.astype(np.float32), q.astype(np.float32),
                       rng.random(T).astype(np.float32), rng.random(T).astype(np.float32))


def deterministic_case(widths: Sequence[int], vocab: int, seed: int, temperature: float = 1.0,
                       logit_std: float = 2.0, peak: Optional[float] = None, peak_rate: float = 0.8,
                       draft_noise: float = 1.0, dup_rate: float = 0.1) -> SampledCase:
    """A draft tree chosen without drawing, as a top-k expansion chooses it,
    with the inputs the stochastic acceptance reads (q is None).

    Target logits are i.i.d. N(0, logit_std^2), and at a share peak_rate of
    the nodes one random token gets `peak` added (default log(vocab) + 5: a
    confident target, so that children are accepted).  A node's children take, in order, the tokens of
    largest logits / temperature + N(0, draft_noise^2) (a drafter correlated
    with the target); each child after the first repeats its previous
    sibling's token with probability dup_rate.  The shape is `random_tree`'s."""
    shape, rng = random_tree(widths, vocab, seed)
    T = shape.n
    peak = math.log(vocab) + 5.0 if peak is None else peak
    logits = rng.normal(0.0, logit_std, size=(T, vocab))
    for u in range(T):
        if rng.random() < peak_rate:
            logits[u, int(rng.integers(0, vocab))] += peak
    z = logits / temperature + rng.normal(0.0, draft_noise, size=(T, vocab))
    tokens = np.zeros(T, dtype=np.int32)
    tokens[0] = rng.integers(0, vocab)
    for u in range(T):
        kids = [c for c in range(1, T) if shape.parents[c] == u]
        if kids:
            order = np.argsort(-z[u], kind="stable")
            for j, c in enumerate(kids):
                tokens[c] = int(order[j])
                if j > 0 and rng.random() < dup_rate:
                    tokens[c] = tokens[kids[j - 1]]
    return SampledCase(Tree(tokens, shape.parents.copy()), logits.astype(np.float32), None,
                       rng.random(T).astype(np.float32), rng.random(T).astype(np.float32))


def workload_tree(w: Workload, index: int, seq: int = 0) -> tuple[Tree, List[int]]:
    """The tree and the node path chosen for planting (possibly empty).

    The planted tokens themselves are the target's greedy continuation, which
    the caller computes and writes with `apply_plant`.
    """
    widths = w.widths_of(seq)
    tree, rng = random_tree(widths, w.model.vocab, tree_seed(w, index, seq))
    if tree.n == 1:
        return tree, []
    children = np.zeros(tree.n, dtype=np.int32)
    for i in range(1, tree.n):
        children[tree.parents[i]] += 1
    if w.plant == "leaf":
        leaves = [i for i in range(1, tree.n) if children[i] == 0]
        leaf = leaves[int(rng.integers(0, len(leaves)))]
        return tree, tree.root_path(leaf)
    if w.plant == "half":
        if rng.random() >= 0.5:
            return tree, []
        depth = tree.depths()
        deepest = [i for i in range(1, tree.n) if depth[i] == len(widths)]
        node = deepest[int(rng.integers(0, len(deepest)))]
        length = int(rng.integers(0, len(widths) + 1))
        return tree, tree.root_path(node)[:length]
    if w.plant == "none":
        return tree, []
    raise ValueError(w.plant)


def apply_plant(tree: Tree, path: Sequence[int], greedy: Sequence[int]) -> Tree:
    """Write greedy[k] into the token of path[k] (path[k] sits at depth k+1)."""
    t = tree.copy()
    for k, node in enumerate(path):
        t.tokens[node] = int(greedy[k])
    return t


def chain_tree(root_token: int, tokens: Sequence[int]) -> Tree:
    T = 1 + len(tokens)
    toks = np.array([root_token, *tokens], dtype=np.int32)
    parents = np.arange(-1, T - 1, dtype=np.int32)
    return Tree(toks, parents)
