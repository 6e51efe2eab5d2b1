"""Stochastic (temperature > 0) acceptance on the GPU, through the C ABI.

Parity with the fp64 oracle (oracle/sampling.py) on the same seeded inputs:
a decision taken in fp32 on the device and in fp64 by the oracle can only
differ when it lies within rounding of its boundary.  So the accepted path is
compared exactly when every accept test on the oracle's path clears
ACCEPT_MARGIN (else the sequence is counted, not compared), and the drawn
token exactly when it clears DRAW_MARGIN, else it must be a valid draw within
DRAW_TOL.  Also: losslessness of the
device walk (chi-square against the exact enumeration of
tests/test_oracle_sampling.py), the small-temperature limit equals the greedy
walk, and the error paths.  Every case prints its name before touching the
GPU.
"""

from collections import defaultdict

import numpy as np
import pytest
import torch

import oracle
from workloads import gen
from tests import test_oracle_sampling as S

pytestmark = pytest.mark.gpu

# An accept test is compared exactly when |u - a| clears ACCEPT_MARGIN; the
# drawn token when u * sum lies DRAW_MARGIN (fraction of the sum) inside its
# interval, and otherwise it must be a token whose interval comes within
# DRAW_TOL of u * sum (fp32 sums over up to 128K terms on the device).
ACCEPT_MARGIN = 1e-5
DRAW_MARGIN = 2e-5
DRAW_TOL = 1e-4


def say(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _lib():
    import paper_2502_11018_amd as P
    return P


def _pack(cases, max_tree, V):
    B = len(cases)
    lg = np.zeros((B * max_tree, V), np.float32)
    q = np.zeros((B * max_tree, V), np.float32)
    ua = np.zeros((B, max_tree), np.float32)
    uf = np.zeros((B, max_tree), np.float32)
    for b, c in enumerate(cases):
        n = c.tree.n
        lg[b * max_tree: b * max_tree + n] = c.logits
        if c.q is not None:
            q[b * max_tree: b * max_tree + n] = c.q
        ua[b, :n] = c.u_accept
        uf[b, :n] = c.u_final
    qd = None if all(c.q is None for c in cases) else torch.from_numpy(q).cuda()
    return torch.from_numpy(lg).cuda(), qd, ua, uf


def _compare(tree, logits, q, ua, uf, T, dev, b, accept_margin=ACCEPT_MARGIN, draw_margin=DRAW_MARGIN,
             draw_tol=DRAW_TOL):
    """Compare device row b with the oracle.  Returns (compared, oracle
    result): False when an accept test on the oracle's path is within
    accept_margin of its boundary (nothing asserted)."""
    tr = []
    r = oracle.accept_sampled(tree, np.asarray(logits, np.float64), None if q is None else np.asarray(q, np.float64),
                              ua, uf, T, tr)
    if any(abs(e[1]) <= accept_margin for e in tr if e[0] == "accept"):
        return False, r
    L = int(dev.length[b])
    assert L == r.length and list(dev.path[b, :L]) == r.path, (b, r, dev.path[b])
    assert list(dev.tokens[b, :L]) == r.tokens[:-1]
    assert all(dev.tokens[b, L + 1:] == -1) and all(dev.path[b, L:] == -1)
    _, margin, rr, cdf = [e for e in tr if e[0] == "draw"][0]
    g = int(dev.tokens[b, L])
    if margin > draw_margin:
        assert g == r.tokens[-1], (b, g, r.tokens[-1], margin)
    else:  # a boundary case: the device token must be a valid draw at u
        lo = cdf[g - 1] if g > 0 else 0.0
        assert lo - draw_tol <= rr <= cdf[g] + draw_tol, (b, g, r.tokens[-1], rr, lo, cdf[g])
    return True, r


@pytest.mark.parametrize("V,T,B", [(3000, 1.0, 8), (128256, 1.0, 3), (3000, 0.7, 8)])
def test_sampled_walk_matches_oracle(V, T, B):
    P = _lib()
    max_tree, D = 64, 6
    cases = [gen.sampled_case((10,) * 6, V, 500 + 17 * i, temperature=T) for i in range(B)]
    lg, q, ua, uf = _pack(cases, max_tree, V)
    say(f"sampled walk V={V} T={T} B={B}")
    res = P.accept_sampled_walk([c.tree for c in cases], lg, q, ua, uf, T, max_tree, D, V)
    compared, lengths = 0, []
    for b, c in enumerate(cases):
        ok, r = _compare(c.tree, c.logits, c.q, c.u_accept, c.u_final, T, res, b)
        compared += ok
        lengths.append(r.length)
    say(f"sampled walk V={V} T={T}: compared {compared}/{B}, oracle lengths {lengths}")
    assert compared >= B - 1


@pytest.mark.parametrize("V,T,B", [(3000, 1.0, 8), (128256, 1.0, 3), (3000, 0.7, 8), (4001, 1.0, 4)])
def test_point_mass_walk_matches_oracle(V, T, B):
    """Deterministic drafts (q_draft NULL): trees whose children are the
    draft's ranked tokens, some repeated, under confident targets so that
    paths are accepted; the odd vocabulary takes the unvectorised loads."""
    P = _lib()
    max_tree, D = 64, 6
    cases = [gen.deterministic_case((10,) * 6, V, 900 + 13 * i, temperature=T) for i in range(B)]
    lg, q, ua, uf = _pack(cases, max_tree, V)
    assert q is None
    say(f"point-mass walk V={V} T={T} B={B}")
    res = P.accept_sampled_walk([c.tree for c in cases], lg, None, ua, uf, T, max_tree, D, V)
    compared, lengths = 0, []
    for b, c in enumerate(cases):
        ok, r = _compare(c.tree, c.logits, None, c.u_accept, c.u_final, T, res, b)
        compared += ok
        lengths.append(r.length)
    say(f"point-mass walk V={V} T={T}: compared {compared}/{B}, oracle lengths {lengths}")
    assert compared >= B - 1
    assert max(lengths) >= 2  # the cases do accept paths


@pytest.mark.parametrize("rule", ["dynamic", "dup"])
def test_point_mass_walk_is_lossless_on_gpu(rule):
    """One deterministic tree (value-dependent branching, or a repeated
    sibling token), accepted 20000 times on the device with fresh uniforms:
    the emitted sequences, extended by target sampling, follow the exact
    enumeration of tests/test_oracle_sampling.py (which equals target
    sampling)."""
    P = _lib()
    D = 2
    Ptab, Qtab = S._tables(6, D)
    exact = S._extend(Ptab, S._exact_point(Ptab, Qtab, (), D, rule), D + 1)
    tree, prefixes = S._det_tree(Qtab, 0, D, rule)
    n, max_tree = 20000, 16
    assert tree.n <= max_tree
    lg = np.zeros((n * max_tree, S.V), np.float32)
    rows = np.stack([np.log(Ptab[pre]) for pre in prefixes]).astype(np.float32)
    for i in range(n):
        lg[i * max_tree: i * max_tree + tree.n] = rows
    rng = np.random.default_rng(31)
    ua = rng.random((n, max_tree)).astype(np.float32)
    uf = rng.random((n, max_tree)).astype(np.float32)
    say(f"point-mass walk losslessness ({rule}): {n} walks of a {tree.n}-node tree")
    res = P.accept_sampled_walk([tree] * n, torch.from_numpy(lg).cuda(), None, ua, uf, 1.0, max_tree, D, S.V)
    counts = defaultdict(int)
    for i in range(n):
        L = int(res.length[i])
        seq = tuple(int(t) for t in res.tokens[i, : L + 1])
        while len(seq) < D + 1:
            seq = seq + (int(rng.choice(S.V, p=Ptab[seq])),)
        counts[seq] += 1
    chi2 = sum((counts[s] - n * e) ** 2 / (n * e) for s, e in exact.items() if e > 0)
    dof = sum(1 for e in exact.values() if e > 0) - 1
    say(f"point-mass walk losslessness ({rule}): chi2 {chi2:.1f} dof {dof}")
    assert chi2 < dof + 6 * np.sqrt(2 * dof), (chi2, dof)


def test_sampled_walk_is_lossless_on_gpu():
    """Trees drawn from a draft table, accepted on the device: the emitted
    sequences, extended by target sampling, follow the exact enumeration
    (which equals target sampling)."""
    P = _lib()
    shape = S.SHAPES[1]
    D = S._depth(shape)
    Ptab, Qtab = S._tables(5, D)
    exact = S._extend(Ptab, S._exact(Ptab, Qtab, (), shape), D + 1)
    rng = np.random.default_rng(21)
    n, max_tree = 20000, 8
    trees, lg, q = [], np.zeros((n * max_tree, S.V), np.float32), np.full((n * max_tree, S.V), 1.0 / S.V, np.float32)
    for i in range(n):
        tokens, parents, prefixes = [int(rng.integers(S.V))], [-1], [()]
        frontier = [(0, shape)]
        while frontier:
            nxt = []
            for node, sh in frontier:
                draws = rng.choice(S.V, size=len(sh), replace=False, p=Qtab[prefixes[node]])
                for t, csh in zip(draws, sh):
                    tokens.append(int(t))
                    parents.append(node)
                    prefixes.append(prefixes[node] + (int(t),))
                    nxt.append((len(tokens) - 1, csh))
            frontier = nxt
        trees.append(gen.Tree(np.array(tokens, np.int32), np.array(parents, np.int32)))
        for j, pre in enumerate(prefixes):
            lg[i * max_tree + j] = np.log(Ptab[pre])
            q[i * max_tree + j] = Qtab[pre]
    ua = rng.random((n, max_tree)).astype(np.float32)
    uf = rng.random((n, max_tree)).astype(np.float32)
    say(f"sampled walk losslessness: {n} trees")
    res = P.accept_sampled_walk(trees, torch.from_numpy(lg).cuda(), torch.from_numpy(q).cuda(), ua, uf, 1.0,
                                max_tree, D, S.V)
    counts = defaultdict(int)
    for i in range(n):
        L = int(res.length[i])
        seq = tuple(int(t) for t in res.tokens[i, : L + 1])
        while len(seq) < D + 1:
            seq = seq + (int(rng.choice(S.V, p=Ptab[seq])),)
        counts[seq] += 1
    chi2 = sum((counts[s] - n * e) ** 2 / (n * e) for s, e in exact.items() if e > 0)
    dof = sum(1 for e in exact.values() if e > 0) - 1
    say(f"sampled walk losslessness: chi2 {chi2:.1f} with {dof} degrees of freedom")
    assert chi2 < dof + 6 * np.sqrt(2 * dof)


def test_small_temperature_equals_greedy_walk():
    P = _lib()
    V, max_tree, D, B = 2000, 64, 6, 6
    cases = [gen.sampled_case((6,) * 6, V, 900 + i, temperature=1.0, logit_std=3.0) for i in range(B)]
    lg, q, ua, uf = _pack(cases, max_tree, V)
    say("sampled walk at T = 1e-3 vs greedy walk")
    res = P.accept_sampled_walk([c.tree for c in cases], lg, q, ua, uf, 1e-3, max_tree, D, V)
    pred = np.zeros((B, max_tree), np.int32)
    for b, c in enumerate(cases):
        pred[b, : c.tree.n] = np.argmax(c.logits, axis=1)
    ref = P.accept_walk([c.tree for c in cases], pred, max_tree, D, V)
    assert (res.length == ref.length).all()
    assert (res.tokens == ref.tokens).all()


def test_sampled_errors():
    P = _lib()
    V, max_tree, D = 100, 16, 4
    c = gen.sampled_case((3, 3), V, 1)
    lg, q, ua, uf = _pack([c], max_tree, V)
    say("sampled walk error paths")
    for T in (0.0, -1.0, float("inf")):
        with pytest.raises(P.GriffinError):
            P.accept_sampled_walk([c.tree], lg, q, ua, uf, T, max_tree, D, V)
    bad = ua.copy()
    bad[0, 1] = 1.0
    with pytest.raises(P.GriffinError):
        P.accept_sampled_walk([c.tree], lg, q, bad, uf, 1.0, max_tree, D, V)


def test_accept_sampled_after_a_step_matches_oracle():
    """The context path: a verify step writes the logits, accept_sampled reads
    them.  The oracle uses its own fp64 logits, so decisions are compared
    where they clear a wider margin (the logits differ by ~1e-5 of their
    range)."""
    P = _lib()
    from tests.test_verify_gpu import Setup
    s = Setup("tiny", n_trees=8)
    try:
        V, T = s.w.model.vocab, 1.0
        rng = np.random.default_rng(33)
        compared = 0
        for i, cases in enumerate(s.cases):
            c = cases[0]
            say(f"accept_sampled after step, tree {i}")
            out = torch.zeros((s.max_tree, V), device="cuda")
            s.v.step([s.w.prefix_len], [c.tree], out)
            q = rng.dirichlet(np.ones(V), size=s.max_tree).astype(np.float32)
            ua = rng.random((1, s.max_tree)).astype(np.float32)
            uf = rng.random((1, s.max_tree)).astype(np.float32)
            res = s.v.accept_sampled(out, torch.from_numpy(q).cuda(), ua, uf, T)
            from tests import harness as H
            ol = H.oracle_sequence(s.ow, c).logits
            ok, _ = _compare(c.tree, ol, q[: c.tree.n], ua[0, : c.tree.n], uf[0, : c.tree.n], T, res, 0,
                             accept_margin=1e-3, draw_margin=1e-3, draw_tol=2e-3)
            compared += ok
        say(f"accept_sampled after step: compared {compared}/8")
        assert compared >= 4
    finally:
        s.v.close()


def test_accept_sampled_before_a_step_is_an_order_error():
    P = _lib()
    from workloads.configs import get_workload
    w = get_workload("tiny")
    mw = gen.make_weights(w.model, 0)
    say("accept_sampled before any step")
    with P.TreeVerifier(w.model, mw.to("cuda"), max_batch=1, max_tree=8, max_depth=7, kv_capacity=64) as v:
        v._batch = 1
        t = torch.zeros((8, w.model.vocab), device="cuda")
        with pytest.raises(P.GriffinError):
            v.accept_sampled(t, t, np.zeros((1, 8)), np.zeros((1, 8)), 1.0)


def test_leaf_rows_of_q_are_not_read():
    """The header's contract: rows of q_draft that belong to leaves are not
    read (NaN there changes nothing), and a NaN logit at the root (always
    visited) is reported as GRIFFIN_ENUMERIC."""
    P = _lib()
    V, max_tree, D, B = 3000, 64, 6, 4
    cases = [gen.sampled_case((10,) * 6, V, 1300 + i) for i in range(B)]
    lg, q, ua, uf = _pack(cases, max_tree, V)
    say("sampled walk: NaN in the q rows of leaves")
    ref = P.accept_sampled_walk([c.tree for c in cases], lg, q, ua, uf, 1.0, max_tree, D, V)
    q2 = q.clone()
    for b, c in enumerate(cases):
        has_kids = set(int(x) for x in c.tree.parents[1:])
        for u in range(c.tree.n):
            if u not in has_kids:
                q2[b * max_tree + u] = float("nan")
    got = P.accept_sampled_walk([c.tree for c in cases], lg, q2, ua, uf, 1.0, max_tree, D, V)
    assert (got.length == ref.length).all() and (got.tokens == ref.tokens).all() and (got.path == ref.path).all()
    say("sampled walk: NaN logit at the root")
    lg2 = lg.clone()
    lg2[0, 17] = float("nan")
    with pytest.raises(P.GriffinError):
        P.accept_sampled_walk([c.tree for c in cases], lg2, q, ua, uf, 1.0, max_tree, D, V)


def _sampled_draft(ow, cache, prefix_len, root, widths, V, T, rng, noise=0.5):
    """A draft tree as a sampling drafter builds it: each expanded node's
    children are drawn without replacement from q = the target's distribution
    at that node (the oracle's, over the tree built so far) perturbed by
    exp(N(0, noise^2)); the first child of each expanded node is expanded
    next.  Returns the tree and q [n, V] (uniform rows at leaves, not read)."""
    tokens, parents, q_rows = [root], [-1], {}
    expand = [0]
    for w in widths:
        lg = oracle.verify_tree(ow, lambda l: (cache.K[l], cache.V[l]),
                                gen.Tree(np.array(tokens, np.int32), np.array(parents, np.int32)),
                                prefix_len).logits
        nxt = []
        for u in expand:
            z = lg[u] / T + rng.normal(0.0, noise, size=V)
            q = np.exp(z - z.max())
            q /= q.sum()
            q_rows[u] = q
            kids = rng.choice(V, size=w, replace=False, p=q)
            first = len(tokens)
            for t in kids:
                tokens.append(int(t))
                parents.append(u)
            nxt.append(first)
        expand = nxt
    n = len(tokens)
    q = np.full((n, V), 1.0 / V)
    for u, row in q_rows.items():
        q[u] = row
    return gen.Tree(np.array(tokens, np.int32), np.array(parents, np.int32)), q


def test_sampled_loop_commits_the_sampled_path():
    """Cycles of step / accept_sampled / commit at T = 1: each commit must move
    the stochastic acceptance's path (not the greedy walk's) into the cache.
    The oracle keeps its own causal cache of every emitted token (the cache
    is bf16 on both sides) and verifies each new tree from it: every cycle's
    logits must match it, and every cycle's decisions must equal the oracle's
    where they clear their margins (else the oracle follows the device's
    valid choice)."""
    from tests.test_verify_gpu import Setup
    from tests import harness as H
    N_TOK, T = 24, 1.0
    s = Setup("tiny", n_trees=1, kv_extra=N_TOK + 16)
    try:
        m = s.w.model
        V = m.vocab
        rng = np.random.default_rng(41)
        cache = s.kvs[0].decode_cache(m)
        P_len = s.w.prefix_len
        root = int(s.cases[0][0].tree.tokens[0])
        emitted, compared, cycles, moved = [], 0, 0, 0
        while len(emitted) < N_TOK:
            tree, q = _sampled_draft(s.ow, cache, P_len, root, (3, 2, 2, 2), V, T, rng)
            ua = rng.random((1, s.max_tree)).astype(np.float32)
            uf = rng.random((1, s.max_tree)).astype(np.float32)
            qd = np.zeros((s.max_tree, V), np.float32)
            qd[: tree.n] = q
            say(f"sampled loop: cycle {cycles} prefix {P_len} nodes {tree.n}")
            out = torch.zeros((s.max_tree, V), device="cuda")
            s.v.step([P_len], [tree], out)
            res = s.v.accept_sampled(out, torch.from_numpy(qd).cuda(), ua, uf, T)
            s.v.commit()
            ol = oracle.verify_tree(s.ow, lambda l: (cache.K[l], cache.V[l]), tree, P_len).logits
            gl = out[: tree.n].cpu().numpy().astype(np.float64)
            rel = (np.abs(gl - ol).max(axis=1) / (ol.max(axis=1) - ol.min(axis=1))).max()
            assert rel < H.REGRESS_REL_TOL, f"cycle {cycles}: logits off by {rel:.2e} of the range"
            ok, _ = _compare(tree, ol, q, ua[0, : tree.n], uf[0, : tree.n], T, res, 0,
                             accept_margin=1e-3, draw_margin=1e-3, draw_tol=2e-3)
            compared += ok
            L, toks, path = res.sequence(0)
            assert [int(tree.tokens[n]) for n in path] == toks[:L]
            moved += L >= 2 or (L == 1 and path[0] != 1)   # a commit the greedy buffer would get wrong
            # the oracle's cache follows: root and accepted tokens, stored as bf16
            for k, t in enumerate([root] + toks[:L]):
                oracle.decode_step(s.ow, cache, int(t), P_len + k)
                for l in range(m.n_layers):
                    cache.K[l][:, -1] = H.bf16_round(cache.K[l][:, -1])
                    cache.V[l][:, -1] = H.bf16_round(cache.V[l][:, -1])
            emitted += toks
            P_len += L + 1
            root = toks[-1]
            cycles += 1
        say(f"sampled loop: {cycles} cycles, {len(emitted)} tokens, decisions compared {compared}/{cycles}, "
            f"commits of a non-trivial sampled path {moved}")
        assert compared >= cycles - 2 and moved >= 2
    finally:
        s.v.close()
