"""Greedy prediction and the acceptance walk.

At temperature 0 (Sec. 5) the target's prediction at a node is the argmax of
its logits.  A draft token is accepted when it equals the target's prediction
at its parent, and a rejected token discards every token after it on that
branch (Sec. 4.1); with a tree, other branches are still tried (Sec. 4.1, the
top-k tree).  The accepted sequence is therefore the deepest node whose whole
root path is accepted, followed by the target's own prediction at that node;
the acceptance length the paper reports (Sec. 5) counts that extra token.

Readings: argmax ties go to the lowest token id; among equally deep accepted
nodes the smallest node id is reported (the accepted tokens are the same for
all of them).
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import List, Sequence

import numpy as np


def argmax_first(logits: np.ndarray) -> np.ndarray:
    """Index of the largest logit per row; the first index wins ties."""
    return np.argmax(logits, axis=-1)


def top2_margin(logits: np.ndarray) -> np.ndarray:
    """Largest minus second-largest logit per row."""
    part = np.partition(logits, -2, axis=-1)
    return part[..., -1] - part[..., -2]


@dataclass
class AcceptResult:
    length: int            # accepted draft tokens L (the paper's tau is L + 1)
    tokens: List[int]      # L draft tokens, then the target's next token
    path: List[int]        # node ids of the L accepted draft tokens


def accept_dfs(tree, pred: Sequence[int]) -> AcceptResult:
    """Depth-first walk from the root along children whose token equals the
    parent's prediction; the deepest visited node (smallest id on ties) wins."""
    T = tree.n
    children: List[List[int]] = [[] for _ in range(T)]
    for i in range(1, T):
        children[int(tree.parents[i])].append(i)
    depth = tree.depths()
    best = 0
    stack = [0]
    while stack:
        n = stack.pop()
        for c in children[n]:
            if int(tree.tokens[c]) == int(pred[n]):
                stack.append(c)
                if depth[c] > depth[best] or (depth[c] == depth[best] and c < best):
                    best = c
    path = tree.root_path(best)
    toks = [int(tree.tokens[i]) for i in path] + [int(pred[best])]
    return AcceptResult(len(path), toks, path)


def accept_trie(tree, greedy: Sequence[int]) -> int:
    """Closed form: the largest l such that some depth-l node carries exactly
    greedy[0..l-1] on its root path (greedy = the target's own continuation)."""
    best = 0
    for i in range(1, tree.n):
        path = tree.root_path(i)
        if len(path) <= len(greedy) and all(int(tree.tokens[n]) == int(greedy[k])
                                            for k, n in enumerate(path)):
            best = max(best, len(path))
    return best
