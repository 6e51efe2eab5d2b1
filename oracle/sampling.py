"""Stochastic tree acceptance at temperature T > 0, in fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper evaluates T in {0, 1} (Sec. 5, experimental setup) and states that
the method is lossless like the speculative-decoding methods it builds on; it
does not restate the acceptance rule for T > 0.  Reading taken here: recursive
rejection sampling over the children of a node, in node-id order, where those
children were drawn from the parent's draft distribution q_u without
replacement:

    p <- softmax(logits_u / T),  q <- q_u
    for each child c of u, token t:
        accept c with probability min(1, p(t) / q(t))
        on rejection:  p <- max(p - q, 0), renormalised
                       q <- q with t removed, renormalised
    a child accepted: continue at that child
    none accepted, or u has no children: emit one token drawn from p

The emitted sequence (accepted draft tokens, then the drawn token) then has the
distribution of sampling the target itself token by token; the pins in
``tests/test_oracle_sampling.py`` check exactly that.

Random draws are inputs: ``u_accept[c]`` decides the test at child c (accept
when u < min(1, p(t)/q(t))), ``u_final[u]`` draws the emitted token at node u.
Drawing from a distribution p with uniform r takes the first token v whose
cumulative sum exceeds r * sum(p) (inverse CDF in token order).

Degenerate inputs, read as: a child whose token has q(t) = 0 is accepted when
p(t) > 0 and rejected otherwise (min(1, p/q) with p/0 = +inf); a rejection
whose residual max(p - q, 0) sums to zero (p = q up to rounding, so the
rejection had probability zero) leaves p unchanged.

Deterministic drafts (q_draft None).  A tree built by ranking the draft's
log-probabilities (the EAGLE-2 expansion the paper follows, App. "Draft Tree
Structure") is a function of the draft's output, not a draw from it: given
the draft, each child proposes its token with probability one.  The same rule
with q the point mass at the child's own token then reads

    accept the child with token t with probability p(t)
    on rejection:  p <- p with t removed, renormalised

and stays lossless for any such tree, however many children a node keeps and
however they were chosen, as long as that choice does not see the target's
uniforms (``tests/test_oracle_sampling.py`` pins it by exact enumeration).  A
draw from q with the count of kept children depending on the draw's values
would not: the kept children would no longer be distributed as q.  Duplicate
sibling tokens are harmless (p(t) is already 0 at the second one).
"""

from __future__ import annotations

from typing import Optional, Sequence

import numpy as np

from .accept import AcceptResult


def softmax_t(logits: np.ndarray, temperature: float) -> np.ndarray:
    """Target distribution at temperature T > 0 (fp64, max subtracted)."""
    if not temperature > 0:
        raise ValueError("temperature must be > 0")
    z = np.asarray(logits, dtype=np.float64) / float(temperature)
    z = z - np.max(z)
    e = np.exp(z)
    return e / np.sum(e)


def draw(p: np.ndarray, r: float, trace: Optional[list] = None) -> int:
    """First token whose cumulative probability exceeds r * sum(p).  With a
    trace list, appends ("draw", margin, r, cdf): margin = the distance of
    r * sum(p) from the nearest cumulative boundary of the chosen token, and
    cdf = the cumulative sums, both as fractions of sum(p)."""
    c = np.cumsum(np.asarray(p, dtype=np.float64))
    thr = float(r) * c[-1]
    idx = min(int(np.searchsorted(c, thr, side="right")), len(c) - 1)
    if trace is not None:
        lo = c[idx - 1] if idx > 0 else 0.0
        trace.append(("draw", min(thr - lo, c[idx] - thr) / c[-1], float(r), c / c[-1]))
    return idx


def _children(parents: np.ndarray, n: int, u: int):
    return [c for c in range(1, n) if int(parents[c]) == u]


def accept_sampled(tree, logits: np.ndarray, q_draft: Optional[np.ndarray], u_accept: Sequence[float],
                   u_final: Sequence[float], temperature: float, trace: Optional[list] = None) -> AcceptResult:
    """Recursive rejection sampling down the tree (one sequence).

    tree: tokens [T], parents [T] (node 0 = root).  logits: [T, V] target
    logits at every node.  q_draft: [T, V], row u = the draft distribution
    u's children were drawn from (rows of leaves are not read), or None for
    a deterministic draft (each child a point mass at its own token).  u_accept,
    u_final: [T] uniforms in [0, 1).  Returns the accepted path (L draft
    tokens and their node ids) and the emitted token appended to the tokens.
    With a trace list, every decision appends its margin: ("accept", u - a)
    for each test and the draw's entry (see `draw`)."""
    tokens = np.asarray(tree.tokens)
    parents = np.asarray(tree.parents)
    n = len(tokens)
    node, path = 0, []
    while True:
        p = softmax_t(logits[node], temperature)
        if q_draft is None:
            nxt = None
            for c in _children(parents, n, node):
                t = int(tokens[c])
                a = float(p[t])
                if trace is not None:
                    trace.append(("accept", float(u_accept[c]) - a))
                if float(u_accept[c]) < a:
                    nxt = c
                    break
                res = p.copy()
                res[t] = 0.0
                if np.sum(res) > 0:
                    p = res / np.sum(res)
            if nxt is None:
                emitted = draw(p, u_final[node], trace)
                break
            path.append(nxt)
            node = nxt
            continue
        q = np.asarray(q_draft[node], dtype=np.float64).copy()
        q = q / np.sum(q) if np.sum(q) > 0 else q
        nxt = None
        for c in _children(parents, n, node):
            t = int(tokens[c])
            if q[t] > 0:
                a = min(1.0, p[t] / q[t])
            else:
                a = 1.0 if p[t] > 0 else 0.0
            if trace is not None:
                trace.append(("accept", float(u_accept[c]) - a))
            if float(u_accept[c]) < a:
                nxt = c
                break
            res = np.maximum(p - q, 0.0)
            if np.sum(res) > 0:
                p = res / np.sum(res)
            q[t] = 0.0
            if np.sum(q) > 0:
                q = q / np.sum(q)
        if nxt is None:
            emitted = draw(p, u_final[node], trace)
            break
        path.append(nxt)
        node = nxt
    return AcceptResult(len(path), [int(tokens[c]) for c in path] + [emitted], path)
