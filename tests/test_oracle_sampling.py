"""Pins of the T > 0 acceptance oracle (oracle/sampling.py) to mathematics it
does not share with itself.

* Losslessness (the property the paper relies on, Sec. 5): an exact
  enumeration, written here independently of the oracle, of the distribution
  of the emitted sequence when every node's children are drawn from the draft
  distribution without replacement and accepted by recursive rejection
  sampling.  Extended by the target's own sampling to a fixed length, it must
  equal sampling the target token by token.  Dropping the renormalisation of
  the residual, or keeping a rejected token in q (on a tree whose rejected
  siblings have children), breaks this equality.
* The uniform-driven oracle, run many times on freshly drawn trees, matches
  that exact distribution (chi-square).
* T -> 0 reduces to the greedy walk; a draft equal to the target accepts every
  first child; drawing reduces to an explicit inverse-CDF loop.
"""

import itertools
from collections import defaultdict

import numpy as np
import pytest

import oracle
from workloads import gen

V = 3


def _tables(seed, depth):
    """Target and draft next-token distributions for every prefix up to depth."""
    rng = np.random.default_rng(seed)
    P, Q = {}, {}
    for d in range(depth + 2):
        for pre in itertools.product(range(V), repeat=d):
            P[pre] = rng.dirichlet(np.full(V, 0.7))
            Q[pre] = rng.dirichlet(np.full(V, 0.7))
    return P, Q


def _norm(x):
    s = x.sum()
    return x / s if s > 0 else x


def _exact(P, Q, prefix, shape):
    """Distribution of the emitted sequence below `prefix`.  shape: tuple of
    child shapes (one entry per child, in draw order; () = no children)."""
    p0, q0 = P[prefix], Q[prefix]
    out = defaultdict(float)
    k = len(shape)
    if k == 0:
        for v in range(V):
            out[(v,)] += p0[v]
        return out
    for draws in itertools.permutations(range(V), k):
        # probability of this ordered draw without replacement from q
        w, left = 1.0, 1.0
        for t in draws:
            w *= q0[t] / left
            left -= q0[t]
        reach, p, q = 1.0, p0.copy(), q0.copy()
        for i, t in enumerate(draws):
            a = min(1.0, p[t] / q[t]) if q[t] > 0 else (1.0 if p[t] > 0 else 0.0)
            for seq, pr in _exact(P, Q, prefix + (t,), shape[i]).items():
                out[(t,) + seq] += w * reach * a * pr
            reach *= 1.0 - a
            r = np.maximum(p - q, 0.0)
            if r.sum() > 0:
                p = r / r.sum()
            q = q.copy()
            q[t] = 0.0
            q = _norm(q)
        for v in range(V):
            out[(v,)] += w * reach * p[v]
    return out


def _extend(P, dist, length):
    """Extend every emitted sequence to `length` tokens by target sampling."""
    out = defaultdict(float)
    for seq, pr in dist.items():
        tails = [((), 1.0)]
        for _ in range(length - len(seq)):
            tails = [(t + (v,), w * P[seq + t][v]) for t, w in tails for v in range(V)]
        for t, w in tails:
            out[seq + t] += pr * w
    return out


SHAPES = [
    ((), ()),                    # root with two leaf children
    (((), ()), ((),)),           # depth 2: 2 children with 2 and 1 children
    (((),), ((),), ((),)),       # three children (all tokens), one grandchild each
    ((((),),),),                 # a chain of depth 3
]


def _depth(shape):
    return 0 if not shape else 1 + max(_depth(c) for c in shape)


@pytest.mark.parametrize("si", range(len(SHAPES)))
@pytest.mark.parametrize("seed", [0, 1])
def test_exact_enumeration_is_lossless(si, seed):
    shape = SHAPES[si]
    D = _depth(shape)
    P, Q = _tables(seed, D)
    ext = _extend(P, _exact(P, Q, (), shape), D + 1)
    assert abs(sum(ext.values()) - 1.0) < 1e-12
    for seq in itertools.product(range(V), repeat=D + 1):
        target = np.prod([P[seq[:k]][seq[k]] for k in range(D + 1)])
        assert abs(ext[seq] - target) < 1e-12, (seq, ext[seq], target)


def _exact_mutated(P, Q, prefix, shape, mutation):
    """The enumeration above with one plausible mistake in the rejection step."""
    p0, q0 = P[prefix], Q[prefix]
    out = defaultdict(float)
    if not shape:
        for v in range(V):
            out[(v,)] += p0[v]
        return out
    for draws in itertools.permutations(range(V), len(shape)):
        w, left = 1.0, 1.0
        for t in draws:
            w *= q0[t] / left
            left -= q0[t]
        reach, p, q = 1.0, p0.copy(), q0.copy()
        for i, t in enumerate(draws):
            a = min(1.0, p[t] / q[t])
            for seq, pr in _exact_mutated(P, Q, prefix + (t,), shape[i], mutation).items():
                out[(t,) + seq] += w * reach * a * pr
            reach *= 1.0 - a
            r = np.maximum(p - q, 0.0)
            if mutation != "residual not renormalised" and r.sum() > 0:
                p = r / r.sum()
            if mutation != "rejected token kept in q":
                q = q.copy()
                q[t] = 0.0
                q = _norm(q)
        for v in range(V):
            out[(v,)] += w * reach * p[v]
    return out


@pytest.mark.parametrize("mutation", ["rejected token kept in q", "residual not renormalised"])
def test_exact_enumeration_detects_near_misses(mutation):
    """Each mistake breaks losslessness on the tree with two children that
    have children of their own, so the pin above tells the rule apart from
    them.  (Keeping the rejected token in q happens to stay lossless when the
    rejected siblings have no children of their own.)"""
    shape = SHAPES[1]
    D = _depth(shape)
    P, Q = _tables(3, D)
    ext = _extend(P, _exact_mutated(P, Q, (), shape, mutation), D + 1)
    err = max(abs(ext[s] - np.prod([P[s[:k]][s[k]] for k in range(D + 1)]))
              for s in itertools.product(range(V), repeat=D + 1))
    assert err > 1e-3


def _draw_without_replacement(rng, q, k):
    q = q.copy()
    out = []
    for _ in range(k):
        t = oracle.draw(q, rng.random())
        out.append(t)
        q[t] = 0.0
    return out


def _sample_tree(rng, Q, shape):
    """Draw a concrete tree (BFS ids) for a shape, children from q w/o replacement."""
    tokens, parents, prefixes = [int(rng.integers(V))], [-1], [()]
    frontier = [(0, shape)]
    while frontier:
        nxt = []
        for node, sh in frontier:
            draws = _draw_without_replacement(rng, Q[prefixes[node]], len(sh))
            for t, csh in zip(draws, sh):
                tokens.append(t)
                parents.append(node)
                prefixes.append(prefixes[node] + (t,))
                nxt.append((len(tokens) - 1, csh))
        frontier = nxt
    return gen.Tree(np.array(tokens, np.int32), np.array(parents, np.int32)), prefixes


@pytest.mark.parametrize("si", [1, 2])
def test_oracle_monte_carlo_matches_exact_distribution(si):
    shape = SHAPES[si]
    D = _depth(shape)
    P, Q = _tables(5, D)
    exact = _extend(P, _exact(P, Q, (), shape), D + 1)
    rng = np.random.default_rng(11)
    n = 20000
    counts = defaultdict(int)
    T = 1.0
    for _ in range(n):
        tree, prefixes = _sample_tree(rng, Q, shape)
        logits = np.stack([np.log(P[pre]) for pre in prefixes])  # softmax(log p) = p at T = 1
        qd = np.stack([Q[pre] for pre in prefixes])
        res = oracle.accept_sampled(tree, logits, qd, rng.random(tree.n), rng.random(tree.n), T)
        seq = tuple(res.tokens)
        while len(seq) < D + 1:  # extend by target sampling
            seq = seq + (oracle.draw(P[seq], rng.random()),)
        counts[seq] += 1
    chi2 = sum((counts[s] - n * e) ** 2 / (n * e) for s, e in exact.items() if e > 0)
    dof = sum(1 for e in exact.values() if e > 0) - 1
    # far tail of chi-square with `dof` degrees of freedom (mean dof, sd sqrt(2 dof))
    assert chi2 < dof + 6 * np.sqrt(2 * dof), (chi2, dof)


def test_small_temperature_reduces_to_greedy_walk():
    rng = np.random.default_rng(2)
    for trial in range(30):
        Vb = 50
        tree, _ = gen.random_tree((3, 4, 5), Vb, 100 + trial)
        # distinct sibling tokens (as drafts drawn without replacement are)
        toks = tree.tokens.copy()
        for u in range(tree.n):
            kids = [c for c in range(1, tree.n) if tree.parents[c] == u]
            for j, c in enumerate(kids):
                toks[c] = (u * 7 + j * 3) % Vb
        tree = gen.Tree(toks, tree.parents)
        logits = rng.normal(size=(tree.n, Vb)) * 3.0
        # plant greedy matches: some children carry their parent's argmax
        for c in range(1, tree.n):
            if rng.random() < 0.5:
                par = tree.parents[c]
                sib = [s for s in range(1, tree.n) if tree.parents[s] == par and s != c]
                if all(toks[s] != np.argmax(logits[par]) for s in sib):
                    toks[c] = int(np.argmax(logits[par]))
        tree = gen.Tree(toks, tree.parents)
        qd = rng.dirichlet(np.ones(Vb), size=tree.n)
        res = oracle.accept_sampled(tree, logits, qd, rng.random(tree.n), rng.random(tree.n), 1e-4)
        ref = oracle.accept_dfs(tree, oracle.argmax_first(logits))
        assert res.tokens == ref.tokens and res.length == ref.length


def test_draft_equal_to_target_accepts_every_first_child():
    rng = np.random.default_rng(4)
    Vb = 20
    tree, _ = gen.random_tree((2, 3, 3), Vb, 7)
    logits = rng.normal(size=(tree.n, Vb))
    T = 0.8
    qd = np.stack([oracle.softmax_t(l, T) for l in logits])
    u_acc = rng.random(tree.n) * 0.999
    u_fin = rng.random(tree.n)
    res = oracle.accept_sampled(tree, logits, qd, u_acc, u_fin, T)
    node, path = 0, []
    while True:
        kids = [c for c in range(1, tree.n) if tree.parents[c] == node]
        if not kids:
            break
        node = kids[0]
        path.append(node)
    assert res.path == path
    assert res.tokens[-1] == oracle.draw(oracle.softmax_t(logits[node], T), u_fin[node])


def test_draw_is_the_inverse_cdf():
    rng = np.random.default_rng(8)
    for _ in range(200):
        p = rng.random(17) * (rng.random(17) < 0.7)
        if p.sum() == 0:
            continue
        r = rng.random()
        acc, want = 0.0, len(p) - 1
        for v in range(len(p)):
            acc += p[v]
            if acc > r * p.sum():
                want = v
                break
        assert oracle.draw(p, r) == want


# ---- deterministic drafts: every child a point mass at its own token ----------

def _det_children(Q, prefix, depth_left, rule):
    """Children tokens of a node, in node-id order, chosen from the draft's
    table without any randomness (as a top-k expansion chooses them)."""
    if depth_left == 0:
        return []
    q = Q[prefix]
    order = [int(v) for v in np.argsort(-q, kind="stable")]
    if rule == "top2":
        return order[:2]
    if rule == "dynamic":  # how many children depends on the draft's values
        return [v for v in order if q[v] > 0.3] or order[:1]
    if rule == "dup":      # a repeated sibling token
        return [order[0], order[0], order[1]]
    if rule == "all":
        return order
    raise ValueError(rule)


def _exact_point(P, Q, prefix, depth_left, rule, mutation=None):
    """Distribution of the emitted sequence below `prefix` when the children,
    tested one after another, are accepted with probability p(t) of the
    renormalised residual, which loses t on rejection (written out by
    enumerating the outcomes of every test)."""
    p = P[prefix].copy()
    out = defaultdict(float)
    reach = 1.0
    for t in _det_children(Q, prefix, depth_left, rule):
        if mutation == "draft ratio":       # as if the child had been drawn from q
            a = min(1.0, p[t] / Q[prefix][t])
        elif mutation == "residual not renormalised":
            a = P[prefix][t] if p[t] > 0 else 0.0
        else:
            a = p[t]
        for seq, pr in _exact_point(P, Q, prefix + (t,), depth_left - 1, rule, mutation).items():
            out[(t,) + seq] += reach * a * pr
        reach *= 1.0 - a
        if mutation != "rejected token kept":
            p = p.copy()
            p[t] = 0.0
            if p.sum() > 0:
                p = p / p.sum()
    for v in range(V):
        out[(v,)] += reach * p[v]
    return out


def _target_err(P, dist, D):
    ext = _extend(P, dist, D + 1)
    assert abs(sum(ext.values()) - 1.0) < 1e-12
    return max(abs(ext[s] - np.prod([P[s[:k]][s[k]] for k in range(D + 1)]))
               for s in itertools.product(range(V), repeat=D + 1))


@pytest.mark.parametrize("rule", ["top2", "dynamic", "dup", "all"])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_point_mass_enumeration_is_lossless(rule, seed):
    """Any tree chosen from the draft alone, with fixed or value-dependent
    branching and with repeated sibling tokens, emits the target's own
    distribution under the point-mass rule."""
    P, Q = _tables(seed, 3)
    assert _target_err(P, _exact_point(P, Q, (), 3, rule), 3) < 1e-12


@pytest.mark.parametrize("mutation", ["draft ratio", "residual not renormalised", "rejected token kept"])
def test_point_mass_enumeration_detects_near_misses(mutation):
    """Testing a deterministic child against the draft's ratio min(1, p/q), not
    renormalising the residual, or leaving a rejected token in it, each
    change the emitted distribution."""
    P, Q = _tables(3, 2)
    assert _target_err(P, _exact_point(P, Q, (), 2, "top2", mutation), 2) > 1e-3


def _det_tree(Q, root, depth, rule):
    """A concrete tree (BFS ids) of _det_children's choices below `root`."""
    tokens, parents, prefixes = [root], [-1], [()]
    frontier = [0]
    for d in range(depth, 0, -1):
        nxt = []
        for node in frontier:
            for t in _det_children(Q, prefixes[node], d, rule):
                tokens.append(t)
                parents.append(node)
                prefixes.append(prefixes[node] + (t,))
                nxt.append(len(tokens) - 1)
        frontier = nxt
    return gen.Tree(np.array(tokens, np.int32), np.array(parents, np.int32)), prefixes


@pytest.mark.parametrize("rule", ["dynamic", "dup"])
def test_point_mass_oracle_monte_carlo_matches_exact_distribution(rule):
    D = 2
    P, Q = _tables(6, D)
    exact = _extend(P, _exact_point(P, Q, (), D, rule), D + 1)
    tree, prefixes = _det_tree(Q, 0, D, rule)
    logits = np.stack([np.log(P[pre]) for pre in prefixes])
    rng = np.random.default_rng(12)
    n = 20000
    counts = defaultdict(int)
    for _ in range(n):
        res = oracle.accept_sampled(tree, logits, None, rng.random(tree.n), rng.random(tree.n), 1.0)
        seq = tuple(res.tokens)
        while len(seq) < D + 1:
            seq = seq + (oracle.draw(P[seq], rng.random()),)
        counts[seq] += 1
    chi2 = sum((counts[s] - n * e) ** 2 / (n * e) for s, e in exact.items() if e > 0)
    dof = sum(1 for e in exact.values() if e > 0) - 1
    assert chi2 < dof + 6 * np.sqrt(2 * dof), (chi2, dof)


def test_point_mass_on_chains_equals_one_hot_draft_rows():
    """On a chain every node has one child, whose point mass is the one-hot
    row at its token: both forms of the rule take the same decisions."""
    rng = np.random.default_rng(13)
    Vb = 30
    for trial in range(40):
        n = 1 + int(rng.integers(1, 7))
        tree = gen.Tree(rng.integers(0, Vb, n).astype(np.int32), np.arange(-1, n - 1, dtype=np.int32))
        logits = rng.normal(size=(n, Vb)) * 2.0
        qd = np.zeros((n, Vb))
        for c in range(1, n):
            qd[c - 1, tree.tokens[c]] = 1.0
        ua, uf = rng.random(n), rng.random(n)
        a = oracle.accept_sampled(tree, logits, None, ua, uf, 0.7)
        b = oracle.accept_sampled(tree, logits, qd, ua, uf, 0.7)
        assert a.tokens == b.tokens and a.path == b.path


def test_point_mass_small_temperature_reduces_to_greedy_walk():
    rng = np.random.default_rng(14)
    Vb = 40
    for trial in range(30):
        tree, _ = gen.random_tree((3, 2, 3), Vb, 300 + trial)
        logits = rng.normal(size=(tree.n, Vb)) * 3.0
        # distinct sibling tokens, one child of some nodes carrying the parent's argmax
        toks = tree.tokens.copy()
        for u in range(tree.n):
            kids = [c for c in range(1, tree.n) if tree.parents[c] == u]
            best = int(np.argmax(logits[u]))
            others = [v for v in range(Vb) if v != best]
            for j, c in enumerate(kids):
                toks[c] = others[(u * 5 + j) % len(others)]
            if kids and rng.random() < 0.7:
                toks[kids[int(rng.integers(len(kids)))]] = best
        tree = gen.Tree(toks, tree.parents)
        res = oracle.accept_sampled(tree, logits, None, rng.random(tree.n), rng.random(tree.n), 1e-4)
        ref = oracle.accept_dfs(tree, oracle.argmax_first(logits))
        assert res.tokens == ref.tokens and res.length == ref.length
