"""The draft-and-verify cycle of GRIFFIN-style speculative decoding (Sec. 3,
Sec. 4): draft a tree, verify it with the target, keep the accepted path and
the target's extra token, then bring the draft up to date.

Every compute step is a library call; this class only sequences them:

1. ``DraftModel.tree``: a tree per sequence by dynamic expansion, rooted at
   the last emitted token, whose input feature is the target's feature of the
   token before it.
2. ``TreeVerifier.step`` / ``accept`` / ``commit``: the target scores the tree
   in one pass, walks it, and moves the accepted path's K/V into its cache.
   At temperature T > 0 (the paper evaluates T = 1 beside greedy decoding,
   Sec. 5) the walk is ``accept_sampled`` over the step's logits with the
   tree as a deterministic draft (each child a point mass at its token: the
   expansion ranks the draft's log-probabilities, it draws nothing), which
   keeps the emitted tokens distributed as sampling the target itself.
3. ``TreeVerifier.features``: the target's features of the root and of the
   accepted nodes.
4. ``DraftModel.extend``: the draft layer's K/V of the root and the accepted
   tokens, each with the target's feature of the token before it, so that the
   draft's cache follows the target's; the feature of the last accepted node
   becomes the next root's input feature.

Both caches hold the same positions: after a cycle that accepts L drafts,
both have prefix_len + L + 1 entries and the target's extra token is the
next root.
"""

from __future__ import annotations

from typing import List, Sequence

import numpy as np
import torch


class _Tree:
    __slots__ = ("tokens", "parents")

    def __init__(self, tokens, parents):
        self.tokens, self.parents = tokens, parents


class SpeculativeCycle:
    """Speculative decoding with a draft model, greedy (temperature 0) or
    sampled (temperature > 0).

    verifier: a ``TreeVerifier`` of the target; draft: a ``DraftModel`` of the
    same target, both on one stream, whose caches hold the same prefix;
    k, depth, n_total: the expansion (the paper's: 10, 6, 60); temperature:
    the target's sampling temperature; seed: the generator of the acceptance
    uniforms when a cycle is not handed its own."""

    def __init__(self, verifier, draft, k: int, depth: int, n_total: int, temperature: float = 0.0,
                 seed: int = 0):
        if draft.max_tree < max(n_total + 1, depth + 1):
            raise ValueError("the draft's max_tree must hold n_total + 1 nodes and a chain of depth + 1 tokens")
        if verifier.max_tree < n_total + 1:
            raise ValueError("the verifier's max_tree must hold n_total + 1 nodes")
        if not (temperature >= 0.0 and np.isfinite(temperature)):
            raise ValueError("temperature must be finite and >= 0")
        self.v, self.d = verifier, draft
        self.k, self.depth, self.n_total = k, depth, n_total
        self.temperature = float(temperature)
        self.rng = np.random.default_rng(seed)
        self.logits = None
        if self.temperature > 0:
            self.logits = torch.empty((verifier.max_batch * verifier.max_tree, verifier.shape.vocab),
                                      dtype=torch.float32, device=verifier.k_cache.device)
        self.prefix: List[int] = []
        self.roots: List[int] = []
        self.root_features = None
        self.last_tree_nodes: List[int] = []
        self.last_accepted: List[int] = []
        self.last_trees: List[_Tree] = []

    def start(self, prefix_len: Sequence[int], roots: Sequence[int], root_features: torch.Tensor):
        """prefix_len[b] tokens cached by both models, roots[b] the next token
        (not cached), root_features [B, d] the target's feature of the token
        before it (CUDA float32)."""
        self.prefix = [int(p) for p in prefix_len]
        self.roots = [int(r) for r in roots]
        self.root_features = root_features.contiguous()

    def cycle(self, uniforms=None) -> List[List[int]]:
        """One cycle; returns the tokens emitted per sequence (the accepted
        drafts, then the target's token after them).  uniforms: at
        temperature > 0, the acceptance's (u_accept, u_final), each
        [B, verifier.max_tree] in [0, 1); drawn from the cycle's generator
        when None."""
        B, T, dm = len(self.roots), self.d.max_tree, self.d.shape.d_model
        n, tok, par, _ = self.d.tree(self.prefix, self.roots, self.root_features, self.k, self.depth, self.n_total)
        trees = [_Tree(tok[b, : n[b]].copy(), par[b, : n[b]].copy()) for b in range(B)]
        self.last_trees = trees
        if self.temperature > 0:
            self.v.step(self.prefix, trees, logits_out=self.logits)
            if uniforms is None:
                shape = (B, self.v.max_tree)
                uniforms = (self.rng.random(shape, dtype=np.float32), self.rng.random(shape, dtype=np.float32))
            acc = self.v.accept_sampled(self.logits, None, uniforms[0], uniforms[1], self.temperature)
        else:
            self.v.step(self.prefix, trees)
            acc = self.v.accept()
        self.v.commit()
        seqs = [acc.sequence(b) for b in range(B)]
        width = max(L for L, _, _ in seqs) + 1
        nodes = np.full((B, width), -1, dtype=np.int32)
        for b, (L, _, path) in enumerate(seqs):
            nodes[b, : L + 1] = [0] + path
        feats = self.v.features(nodes)                       # [B, width, d]: root, then the accepted nodes
        ext = torch.zeros((B, T, dm), dtype=torch.float32, device=feats.device)
        ext[:, 0] = self.root_features
        ext[:, 1:width] = feats[:, : width - 1]
        chains = [[self.roots[b]] + toks[:L] for b, (L, toks, _) in enumerate(seqs)]
        self.d.extend(self.prefix, chains, ext)
        last = torch.as_tensor([L for L, _, _ in seqs], device=feats.device)
        self.root_features = feats[torch.arange(B, device=feats.device), last].contiguous()
        out = []
        for b, (L, toks, _) in enumerate(seqs):
            self.prefix[b] += L + 1
            self.roots[b] = toks[-1]
            out.append(toks)
        self.last_tree_nodes = [int(x) for x in n]
        self.last_accepted = [L for L, _, _ in seqs]
        return out
