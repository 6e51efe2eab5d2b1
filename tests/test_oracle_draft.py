"""Pins of the draft-model oracle (oracle/draft.py) to facts it does not
share with itself.

* The reading of the draft's shapes (TGF expansion 11008, TEH two d x d
  heads, one decoder layer of the target's shape) gives the draft of the 8B
  target exactly the parameter count the paper publishes (App., "Parameter
  Sizes of GRIFFIN's Draft Models": 0.42B).
* LayerNorm and TGF reduce to closed forms for special weights.
* With TGF passing the token embedding through unchanged and an identity
  predict head, a draft pass is exactly the pinned one-layer target pass of
  oracle.verify_tree (same layer, prefix and tree).
* Tree attention: tokens outside a node's ancestry leave its outputs unchanged.
* Top-k log-probabilities equal a sort and a log-sum-exp of the full row.
* Expansion: invariants of the result; with nothing truncated (depth 2,
  every token proposed) it equals the brute-force best paths; a hand-worked
  case where ranking by cumulative and by local probability disagree.
"""

import itertools

import numpy as np
import pytest
import torch

import oracle
from oracle import draft as od
from workloads import gen
from workloads.configs import DRAFTS


def test_draft_parameter_count_matches_the_paper():
    # 0.42B for the 8B target (the appendix rounds to two decimals)
    assert round(DRAFTS["llama3-8b"].param_count() / 1e9, 2) == 0.42


def test_layernorm_closed_form():
    rng = np.random.default_rng(0)
    x = rng.normal(size=(5, 64)) * 3 + 2
    g, b = rng.normal(size=64), rng.normal(size=64)
    y = od.layernorm(x, np.ones(64), np.zeros(64), 1e-12)
    assert np.allclose(y.mean(axis=1), 0, atol=1e-12) and np.allclose(y.var(axis=1), 1, atol=1e-9)
    # affine: gain and bias act per column
    assert np.allclose(od.layernorm(x, g, b, 1e-12), y * g + b, atol=1e-12)
    # a constant row maps to the bias (zero variance, eps keeps it finite)
    assert np.allclose(od.layernorm(np.full((1, 64), 7.0), g, b, 1e-5), b)


def _small():
    ds = DRAFTS["tiny"]
    mw = gen.make_weights(ds.target, 0)
    ow = oracle.OracleWeights(mw)
    dw = gen.make_draft_weights(ds, 3)
    return ds, mw, ow, dw


def _kv(ds, P, seed=5):
    k, v = gen.synthetic_kv(ds.layer, 0, 0, P, seed)
    return k.double().numpy(), v.double().numpy()


def test_tgf_closed_forms():
    ds, mw, ow, dw = _small()
    d, e = ds.target.d_model, ds.tgf_dim
    rng = np.random.default_rng(1)
    F, x = rng.normal(size=(3, d)), rng.normal(size=(3, d))
    dow = od.DraftOracleWeights(dw, ow)
    t = dow.t
    t["w_m"] = np.concatenate([np.eye(d), np.zeros((d, d))], axis=1)   # h = F + b_m
    t["w_u"] = np.zeros((e, 2 * d))
    t["b_u"] = np.zeros(e)                                             # z = 0, SiLU(0) = 0
    h, o = od.tgf(dow, F, x)
    assert np.allclose(h, F + t["b_m"]) and np.allclose(o, h + t["b_d"])
    t["w_m"] = np.concatenate([np.zeros((d, d)), np.eye(d)], axis=1)   # h = e + b_m
    t["b_u"] = np.full(e, 2.0)                                         # z = 2 everywhere
    h, o = od.tgf(dow, F, x)
    silu2 = 2.0 / (1.0 + np.exp(-2.0))
    assert np.allclose(h, x + t["b_m"])
    assert np.allclose(o, silu2 * t["w_d"].sum(axis=1) + t["b_d"] + h)


def test_draft_pass_reduces_to_the_target_pass():
    """TGF = the embedding (W_m = [0 | I], SiLU(z) ~ 0), predict head = I: the
    draft pass is the one-layer target pass with the draft's layer."""
    ds, mw, ow, dw = _small()
    d, e = ds.target.d_model, ds.tgf_dim
    dow = od.DraftOracleWeights(dw, ow)
    t = dow.t
    t["w_m"] = np.concatenate([np.zeros((d, d)), np.eye(d)], axis=1)
    t["b_m"] = np.zeros(d)
    t["w_u"] = np.zeros((e, 2 * d))
    t["b_u"] = np.full(e, -60.0)            # SiLU(-60) ~ -5e-25
    t["b_d"] = np.zeros(d)
    t["w_p"], t["b_p"] = np.eye(d), np.zeros(d)
    P = 40
    Kp, Vp = _kv(ds, P)
    tree, _ = gen.random_tree((3, 4, 2), ds.target.vocab, 17)
    feats = np.random.default_rng(2).normal(size=(tree.n, d))
    r = od.draft_forward(dow, tree, feats, (Kp, Vp), P)
    one = gen.ModelWeights(ds.layer, mw.embed, mw.lm_head, mw.final_norm, [dw.layer])
    ref = oracle.verify_tree(oracle.OracleWeights(one), lambda l: (Kp, Vp), tree, P)
    assert np.max(np.abs(r.logits - ref.logits)) < 1e-12 * np.max(np.abs(ref.logits))
    assert np.allclose(r.y, ref.hidden, rtol=0, atol=1e-12)


def test_tokens_outside_the_ancestry_do_not_matter():
    ds, mw, ow, dw = _small()
    dow = od.DraftOracleWeights(dw, ow)
    P = 30
    kv = _kv(ds, P)
    tree, _ = gen.random_tree((3, 3, 3), ds.target.vocab, 4)
    feats = np.random.default_rng(3).normal(size=(tree.n, ds.target.d_model))
    a = od.draft_forward(dow, tree, feats, kv, P)
    anc = od.ancestor_matrix(tree.parents)
    node = tree.n - 1
    other = [j for j in range(tree.n) if not anc[node, j]]
    t2 = tree.copy()
    feats2 = feats.copy()
    for j in other:
        t2.tokens[j] = (t2.tokens[j] + 1) % ds.target.vocab
        feats2[j] += 1.0
    b = od.draft_forward(dow, t2, feats2, kv, P)
    assert np.array_equal(a.logits[node], b.logits[node]) and np.array_equal(a.regress[node], b.regress[node])
    assert not np.allclose(a.logits[other[0]], b.logits[other[0]])


def test_topk_logprobs():
    rng = np.random.default_rng(6)
    lg = rng.normal(size=(4, 50)) * 2
    lg[1, 7] = lg[1, 9] = lg[1].max() + 1.0   # a tie: the lower id first
    tok, lp = od.topk_logprobs(lg, 5)
    assert list(tok[1, :2]) == [7, 9]
    for r in range(4):
        full = lg[r] - np.log(np.sum(np.exp(lg[r])))
        assert np.allclose(np.exp(full).sum(), 1.0)
        assert list(tok[r]) == list(np.argsort(-lg[r], kind="stable")[:5])
        assert np.allclose(lp[r], full[tok[r]])


class _TableDraft:
    """A draft whose next-token distribution is a fixed function of the path
    (seeded per path), on a small vocabulary."""

    def __init__(self, V, seed, k):
        self.V, self.seed, self.k = V, seed, k

    def dist(self, path):
        rng = np.random.default_rng([self.seed, *[t + 1 for t in path]])
        return rng.dirichlet(np.full(self.V, 0.6))

    def step(self, ptree, feats):
        T = ptree.n
        tok = np.zeros((T, self.k), np.int32)
        lp = np.zeros((T, self.k))
        for i in range(T):
            path = tuple(int(ptree.tokens[j]) for j in [0, *ptree.root_path(i)])
            p = self.dist(path)
            order = np.argsort(-p, kind="stable")[: self.k]
            tok[i], lp[i] = order, np.log(p[order])
        return tok, lp, np.zeros((T, 4))


def _paths(tree):
    return {tuple(int(tree.tokens[j]) for j in tree.root_path(i)) for i in range(1, tree.n)}


@pytest.mark.parametrize("seed", range(6))
def test_expansion_invariants(seed):
    V, k, D, N = 7, 3, 4, 10
    td = _TableDraft(V, seed, k)
    ex = od.expand_tree(2, np.zeros(4), td.step, k, D, N, gen.Tree)
    t = ex.tree
    assert t.n == N + 1 and t.parents[0] == -1
    assert all(0 <= t.parents[i] < i for i in range(1, t.n))
    d = t.depths()
    assert d.max() <= D and np.all(np.diff(d) >= 0)
    for i in range(1, t.n):
        assert ex.scores[i] <= ex.scores[t.parents[i]] + 1e-15
    # the kept nodes are the best candidates
    assert ex.scores[1:].min() >= np.sort(ex.candidate_scores)[::-1][N - 1] - 1e-15
    assert len(ex.passes) == D and all(p.n == 1 + k * i for i, p in enumerate(ex.passes))
    # scores are the paths' log-probabilities under the draft
    for i in range(1, t.n):
        path = [int(t.tokens[0])]
        lp = 0.0
        for j in t.root_path(i):
            lp += np.log(td.dist(tuple(path))[int(t.tokens[j])])
            path.append(int(t.tokens[j]))
        assert abs(lp - ex.scores[i]) < 1e-12


@pytest.mark.parametrize("seed", range(4))
def test_untruncated_expansion_is_the_best_paths(seed):
    """Depth 2 with every token proposed and kept: the result is the N most
    probable paths of length 1 or 2, found by enumerating all of them."""
    V, N = 5, 12
    td = _TableDraft(V, 100 + seed, V)
    ex = od.expand_tree(0, np.zeros(4), td.step, V, 2, N, gen.Tree)
    allp = []
    for L in (1, 2):
        for path in itertools.product(range(V), repeat=L):
            lp, pre = 0.0, (0,)
            for tkn in path:
                lp += np.log(td.dist(pre)[tkn])
                pre = pre + (tkn,)
            allp.append((lp, path))
    best = {p for _, p in sorted(allp, key=lambda x: -x[0])[:N]}
    assert _paths(ex.tree) == best


def test_expansion_hand_worked_case():
    """V = 3 tokens {0, 1, 2}, k = 2, depth 3.  Root proposals: 0 (p .5), 1 (.3);
    children of 0: 0 (.4), 1 (.35); children of 1: 0 (.55), 1 (.45).  Depth-2
    cumulative scores: (0,0) .2, (0,1) .175, (1,0) .165, (1,1) .135, so the
    depth-2 nodes expanded in the third pass are (0,0) and (0,1), although the
    children of 1 are more probable given their parent."""
    table = {(): [.5, .3, .2], (0,): [.4, .35, .25], (1,): [.55, .45, 0.0]}

    def step(ptree, feats):
        T = ptree.n
        tok, lp = np.zeros((T, 2), np.int32), np.zeros((T, 2))
        for i in range(T):
            path = tuple(int(ptree.tokens[j]) for j in ptree.root_path(i))
            p = np.array(table.get(path, [.6, .3, .1]))
            order = np.argsort(-p, kind="stable")[:2]
            tok[i], lp[i] = order, np.log(np.maximum(p[order], 1e-300))
        return tok, lp, np.zeros((T, 2))

    ex = od.expand_tree(2, np.zeros(2), step, 2, 3, 4, gen.Tree)
    third = ex.passes[2]
    expanded = {tuple(int(third.tokens[j]) for j in third.root_path(i)) for i in range(1, third.n)}
    assert expanded == {(0,), (1,), (0, 0), (0, 1)}
    # final 4: (0) .5, (1) .3, (0,0) .2, (0,1) .175
    assert _paths(ex.tree) == {(0,), (1,), (0, 0), (0, 1)}
    assert list(ex.tree.parents) == [-1, 0, 0, 1, 1]


def test_chain_kv_extends_the_prefix():
    """A draft pass over a chain adds exactly the chain's K/V to the draft's
    cache: passing the first tokens, appending their K/V to the prefix and
    then passing the last token alone (at its position, with its feature)
    reproduces the last row of the pass over the whole chain."""
    ds, mw, ow, dw = _small()
    dow = od.DraftOracleWeights(dw, ow)
    P, d = 33, ds.target.d_model
    Kp, Vp = _kv(ds, P)
    toks = [7, 100, 3, 512, 9]
    feats = np.random.default_rng(4).normal(size=(len(toks), d))
    whole = od.draft_forward(dow, gen.chain_tree(toks[0], toks[1:]), feats, (Kp, Vp), P)
    head = od.draft_forward(dow, gen.chain_tree(toks[0], toks[1:-1]), feats[:-1], (Kp, Vp), P)
    K2 = np.concatenate([Kp, head.k.transpose(1, 0, 2)], axis=1)
    V2 = np.concatenate([Vp, head.v.transpose(1, 0, 2)], axis=1)
    last = od.draft_forward(dow, gen.chain_tree(toks[-1], []), feats[-1:], (K2, V2), P + len(toks) - 1)
    assert np.allclose(last.logits[0], whole.logits[-1], rtol=0, atol=1e-9)
    assert np.allclose(last.regress[0], whole.regress[-1], rtol=0, atol=1e-9)
    assert np.allclose(head.k, whole.k[:-1], atol=1e-12) and np.allclose(head.v, whole.v[:-1], atol=1e-12)


def test_draft_layer_of_an_moe_target_is_dense():
    """The draft of an MoE target has one dense SwiGLU layer of the experts'
    width: its pass equals that of a draft whose target is the same model made
    dense (the weights are the same tensors)."""
    from dataclasses import replace
    ds = DRAFTS["small-moe"]
    assert ds.layer.n_experts == 1 and ds.layer.d_ff == ds.target.d_ff
    mw = gen.make_weights(ds.target, 0)
    dw = gen.make_draft_weights(ds, 3)
    dense = replace(ds.target, n_experts=1, top_k=1)
    dw_dense = gen.DraftWeights(replace(ds, target=dense), dw.t, dw.layer)
    mw_dense = gen.ModelWeights(dense, mw.embed, mw.lm_head, mw.final_norm, [])
    P = 25
    k, v = gen.synthetic_kv(ds.layer, 0, 0, P, 5)
    kv = (k.double().numpy(), v.double().numpy())
    tree, _ = gen.random_tree((2, 3), ds.target.vocab, 8)
    feats = np.random.default_rng(3).normal(size=(tree.n, ds.target.d_model))
    a = od.draft_forward(od.DraftOracleWeights(dw, oracle.OracleWeights(mw)), tree, feats, kv, P)
    b = od.draft_forward(od.DraftOracleWeights(dw_dense, oracle.OracleWeights(mw_dense)), tree, feats, kv, P)
    assert np.array_equal(a.logits, b.logits) and np.array_equal(a.regress, b.regress)
