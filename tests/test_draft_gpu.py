"""The draft model on the GPU, through the C ABI, against the fp64 oracle
(oracle/draft.py) on the same seeded inputs.

A draft pass: every live row's top-k tokens and log-probabilities.  The
token of a rank is compared exactly where the oracle's logit of that rank
is separated from both neighbouring ranks by more than TOKEN_GAP (fp32 /
split-bf16 on the device, fp64 in the oracle); at every rank the token must
carry that rank's oracle logit within TOKEN_GAP; log-probabilities within
LOGP_TOL.  A drafted tree: the set of root paths
equals the oracle's expansion wherever none of its selections (the
frontier of each depth, the final n_total) is decided by a score gap below
SCORE_GAP; every drafted tree, decided or not, must be a correct expansion
of the oracle's draft (scores, top-k membership, nothing dropped that beats
the kept nodes by more than SCORE_GAP).  Every case prints its name first.
"""

import numpy as np
import pytest
import torch

import oracle
from oracle import draft as od
from workloads import gen
from workloads.configs import DRAFTS

pytestmark = pytest.mark.gpu

TOKEN_GAP = 2e-3
LOGP_TOL = 2e-3
SCORE_GAP = 2e-3


def say(msg):
    print(f"[gpu-case] {msg}", flush=True)


class Draft:
    def __init__(self, name, batch, prefix, max_tree=64):
        import paper_2502_11018_amd as P
        self.ds = DRAFTS[name]
        m = self.ds.target
        self.mw = gen.make_weights(m, 0)
        self.dw = gen.make_draft_weights(self.ds, 3)
        self.ow = oracle.OracleWeights(self.mw)
        self.dow = od.DraftOracleWeights(self.dw, self.ow)
        self.prefix = prefix
        cap = ((max(prefix) + max_tree + 63) // 64) * 64
        say(f"draft {name}: init batch {batch} cap {cap}")
        self.dm = P.DraftModel(self.ds, self.dw.to("cuda"), self.mw.to("cuda"), max_batch=batch, max_tree=max_tree,
                               max_depth=max_tree - 1, kv_capacity=cap)
        self.kv = []
        for b in range(batch):
            k, v = gen.synthetic_kv(self.ds.layer, 0, b, prefix[b], 5)
            self.kv.append((k.double().numpy(), v.double().numpy()))
            self.dm.write_prefix(b, k.cuda(), v.cuda())
        self.feat = gen.draft_root_features(m.d_model, batch, 11)
        torch.cuda.synchronize()

    def close(self):
        self.dm.close()


def _pass_feats(dr, tree, fr_prev, root_feat):
    """Input features of a pass: the root's, then each node's parent's regress feature."""
    f = np.zeros((tree.n, dr.ds.target.d_model))
    f[0] = root_feat
    for i in range(1, tree.n):
        f[i] = fr_prev[tree.parents[i]]
    return f


@pytest.mark.parametrize("name", ["tiny", "small-gqa", "small-moe", "tiny-v20001", "tiny-v20000"])
def test_draft_passes_match_oracle(name):
    """Three passes over growing trees, as an expansion runs them: the root
    alone, then its children, then grandchildren; each node reads its
    parent's regress feature from the previous pass (the oracle's from its
    own fp64 pass).  Top-k tokens and log-probabilities of every node."""
    B = 2
    dr = Draft(name, B, [37, 70])
    try:
        k, V, d = dr.ds.k, dr.ds.target.vocab, dr.ds.target.d_model
        compared, total = 0, 0
        fr_prev = [None] * B
        for it, widths in enumerate([(), (3,), (3, 4)]):
            trees = [gen.random_tree(widths, V, 50 + 7 * b)[0] for b in range(B)]
            say(f"draft {name} pass {it}: {[t.n for t in trees]} nodes")
            tok, lp = dr.dm.step(dr.prefix, trees, dr.feat.cuda(), k)
            for b, t in enumerate(trees):
                feats = np.zeros((t.n, d))
                feats[0] = dr.feat[b].double().numpy()
                for i in range(1, t.n):
                    feats[i] = fr_prev[b][t.parents[i]]
                r = od.draft_forward(dr.dow, t, feats, dr.kv[b], dr.prefix[b])
                fr_prev[b] = r.regress
                otok, _ = od.topk_logprobs(r.logits, k)
                srt = np.sort(r.logits, axis=1)[:, ::-1]
                for i in range(t.n):
                    full = r.logits[i] - (srt[i, 0] + np.log(np.exp(r.logits[i] - srt[i, 0]).sum()))
                    assert np.max(np.abs(lp[b, i] - full[tok[b, i]])) < LOGP_TOL, (b, i)
                    # valid at every rank: distinct tokens, each with its rank's value
                    assert len(set(tok[b, i].tolist())) == k and tok[b, i].min() >= 0 and tok[b, i].max() < V
                    assert np.max(np.abs(r.logits[i][tok[b, i]] - srt[i, :k])) <= TOKEN_GAP, (b, i)
                    # unique where the rank's value is separated from both neighbours
                    gap = -np.diff(srt[i, : k + 1])
                    for j in range(k):
                        total += 1
                        if gap[j] > TOKEN_GAP and (j == 0 or gap[j - 1] > TOKEN_GAP):
                            compared += 1
                            assert tok[b, i, j] == otok[i, j], (b, i, j, tok[b, i], otok[i])
        say(f"draft {name}: tokens compared at {compared}/{total} ranks")
        assert compared >= total // 2
    finally:
        dr.close()


def _decided(ex, k, depth, n_total):
    """True when every selection of the oracle's expansion clears SCORE_GAP:
    the k-th vs (k+1)-th new candidate of each expanded depth, and the
    n_total-th vs (n_total+1)-th candidate overall."""
    sc = ex.candidate_scores
    per = [k] + [k * k] * (depth - 1)
    at = 0
    for t in range(depth - 1):
        new = np.sort(sc[at: at + per[t]])[::-1]
        if len(new) > k and new[k - 1] - new[k] <= SCORE_GAP:
            return False
        at += per[t]
    allc = np.sort(sc)[::-1]
    return not (len(allc) > n_total and allc[n_total - 1] - allc[n_total] <= SCORE_GAP)


def _path_set(n, tok, par):
    out = set()
    for i in range(1, n):
        path, j = [], i
        while j > 0:
            path.append(int(tok[j]))
            j = int(par[j])
        out.add(tuple(path[::-1]))
    return out


def _oracle_scores(dr, b, n, tok, par, D):
    """The oracle's view of a drafted tree: every node's path log-probability
    and every node's full log-softmax row.  A node's outputs depend only on
    its root path (the ancestor mask) and its input feature, its parent's
    regress feature from the previous pass, so D passes over the whole tree
    make every node of depth <= p exact after pass p."""
    t = gen.Tree(np.asarray(tok[:n], np.int32), np.asarray(par[:n], np.int32))
    depth = t.depths()
    feats = np.zeros((n, dr.ds.target.d_model))
    feats[0] = dr.feat[b].double().numpy()
    logp = [None] * n
    prev = None
    for p in range(D):
        if prev is not None:
            for i in range(1, n):
                feats[i] = prev[t.parents[i]]
        r = od.draft_forward(dr.dow, t, feats, dr.kv[b], dr.prefix[b])
        for i in range(n):
            if depth[i] == p:
                row = r.logits[i]
                mx = row.max()
                logp[i] = row - (mx + np.log(np.exp(row - mx).sum()))
        prev = r.regress
    score = np.zeros(n)
    for i in range(1, n):
        score[i] = score[t.parents[i]] + logp[t.parents[i]][t.tokens[i]]
    return t, depth, score, logp


def _check_valid_expansion(dr, b, n, tok, par, sc, k, D, N):
    """A drafted tree that near-ties may have decided differently from the
    oracle's expansion must still be a correct expansion of the oracle's
    draft: each kept node's score is its path log-probability (within
    LOGP_TOL per level), each kept child is one of its parent's top-k
    tokens (within TOKEN_GAP), and no candidate proposed by a node that kept
    children but itself dropped scores above the worst kept node by more than
    SCORE_GAP."""
    t, depth, score, logp = _oracle_scores(dr, b, n, tok, par, D)
    for i in range(1, n):
        assert abs(sc[i] - score[i]) <= LOGP_TOL * depth[i], (b, i, sc[i], score[i])
    worst = min(score[1:])
    kids = {}
    for i in range(1, n):
        kids.setdefault(int(t.parents[i]), []).append(i)
    for u, ch in kids.items():
        top = np.argsort(-logp[u], kind="stable")[:k]
        kth = logp[u][top[-1]]
        kept = {int(t.tokens[c]) for c in ch}
        for c in ch:
            assert logp[u][t.tokens[c]] >= kth - TOKEN_GAP, (b, u, c)
        for v in top:
            if int(v) not in kept:
                assert score[u] + logp[u][v] <= worst + SCORE_GAP, (b, u, int(v), score[u] + logp[u][v], worst)


@pytest.mark.parametrize("name", ["tiny", "small-gqa", "tiny-v20000"])
def test_drafted_tree_matches_oracle_expansion(name):
    B = 3
    dr = Draft(name, B, [20, 61, 90])
    try:
        ds = dr.ds
        k, D, N, d = ds.k, ds.depth, ds.n_total, ds.target.d_model
        roots = [5, 17, 29]
        say(f"draft {name}: tree k={k} depth={D} n_total={N}")
        n, tok, par, sc = dr.dm.tree(dr.prefix, roots, dr.feat.cuda(), k, D, N)
        again = dr.dm.tree(dr.prefix, roots, dr.feat.cuda(), k, D, N)
        assert all(np.array_equal(a, b) for a, b in zip((n, tok, par, sc), again)), "not deterministic"
        compared = 0
        for b in range(B):
            assert n[b] == N + 1 and par[b, 0] == -1
            assert all(0 <= par[b, i] < i for i in range(1, n[b]))

            def step(ptree, feats, b=b):
                r = od.draft_forward(dr.dow, ptree, feats, dr.kv[b], dr.prefix[b])
                tk, lp = od.topk_logprobs(r.logits, k)
                return tk, lp, r.regress

            ex = od.expand_tree(roots[b], dr.feat[b].double().numpy(), step, k, D, N, gen.Tree)
            # valid whatever near-ties decided: scores fall along every path, depth <= D
            assert sc[b, 0] == 0 and all(sc[b, i] <= sc[b, par[b, i]] for i in range(1, n[b]))
            depth = [0] * n[b]
            for i in range(1, n[b]):
                depth[i] = depth[par[b, i]] + 1
            assert max(depth) <= D
            _check_valid_expansion(dr, b, n[b], tok[b], par[b], sc[b], k, D, N)
            if _decided(ex, k, D, N):
                compared += 1
                assert np.max(np.abs(np.sort(sc[b, : n[b]]) - np.sort(ex.scores))) < 1e-2
                assert _path_set(n[b], tok[b], par[b]) == _path_set(ex.tree.n, ex.tree.tokens, ex.tree.parents)
        say(f"draft {name}: trees compared {compared}/{B}")
        assert compared >= 1
    finally:
        dr.close()


def _host_expansion(dm, prefix, roots, feat, k, D, N):
    """The tree expansion written out on the host over single draft passes
    (griffin_draft_step), in fp64 with Python's stable sorts: each pass's
    frontier proposes its top-k, a candidate scores its parent's score plus
    its log-probability, the k best new candidates (ties: the earlier one)
    are the next frontier, and the tree is the N best candidates numbered by
    depth, then rank.  The pass trees are those griffin_draft_tree builds on
    the device, so both see the same top-k values."""
    B = len(roots)
    ptok = [[int(r)] for r in roots]
    ppar = [[-1] for _ in roots]
    pcand = [[-1] for _ in roots]
    pscore = [[0.0] for _ in roots]
    front = [[0] for _ in roots]
    cands = [[] for _ in roots]  # (depth, proposing pass-tree node, token, score)
    for t in range(D):
        trees = [gen.Tree(np.asarray(ptok[b], np.int32), np.asarray(ppar[b], np.int32)) for b in range(B)]
        ktok, klp = dm.step(prefix, trees, feat, k)
        for b in range(B):
            fresh = []
            for r in front[b]:
                for j in range(k):
                    cands[b].append((t + 1, r, int(ktok[b, r, j]), pscore[b][r] + float(klp[b, r, j])))
                    fresh.append(len(cands[b]) - 1)
            if t + 1 == D:
                continue
            fresh.sort(key=lambda i, cb=cands[b]: -cb[i][3])
            front[b] = []
            for i in fresh[:k]:
                _, r, tk, s = cands[b][i]
                ptok[b].append(tk)
                ppar[b].append(r)
                pcand[b].append(i)
                pscore[b].append(s)
                front[b].append(len(ptok[b]) - 1)
    out = []
    for b in range(B):
        cb = cands[b]
        chosen = sorted(range(len(cb)), key=lambda i: -cb[i][3])[:N]
        rank = {c: i for i, c in enumerate(chosen)}
        order = sorted(chosen, key=lambda i: (cb[i][0], rank[i]))
        index = {c: i + 1 for i, c in enumerate(order)}
        tok = [int(roots[b])] + [cb[i][2] for i in order]
        par = [-1] + [0 if pcand[b][cb[i][1]] < 0 else index[pcand[b][cb[i][1]]] for i in order]
        sc = np.asarray([0.0] + [cb[i][3] for i in order]).astype(np.float32)
        out.append((tok, par, sc))
    return out


@pytest.mark.parametrize("name,k,D,N", [("tiny", None, None, None), ("tiny-v20000", None, None, None),
                                        ("tiny", 16, 4, 63), ("tiny", 3, 6, 10), ("tiny", 2, 3, 50),
                                        ("tiny", 1, 5, 3)])
def test_device_expansion_equals_host_expansion_of_its_passes(name, k, D, N):
    """griffin_draft_tree selects on the device; written out on the host over
    the same passes, the selection must give the same tree bit for bit
    (tokens, parents, float32 scores), including n_total above the candidate
    count, the largest k, k = 1 and the single-node frontier of the first pass."""
    B = 3
    dr = Draft(name, B, [20, 61, 90])
    try:
        ds = dr.ds
        k, D, N = k or ds.k, D or ds.depth, N or ds.n_total
        roots = [5, 17, 29]
        feat = dr.feat.cuda()
        say(f"draft {name}: device vs host expansion k={k} depth={D} n_total={N}")
        n, tok, par, sc = dr.dm.tree(dr.prefix, roots, feat, k, D, N)
        ref = _host_expansion(dr.dm, dr.prefix, roots, feat, k, D, N)
        for b in range(B):
            rt, rp, rs = ref[b]
            assert n[b] == len(rt), (b, n[b], len(rt))
            assert tok[b, : n[b]].tolist() == rt, b
            assert par[b, : n[b]].tolist() == rp, b
            assert np.array_equal(sc[b, : n[b]], rs), b
    finally:
        dr.close()


def test_draft_errors():
    import paper_2502_11018_amd as P
    dr = Draft("tiny", 1, [30], max_tree=16)
    try:
        say("draft errors")
        with pytest.raises(P.GriffinError):   # 1 + k (depth - 1) = 1 + 4 * 4 > 16
            dr.dm.tree([30], [1], dr.feat[:1].cuda(), 4, 5, 12)
        with pytest.raises(P.GriffinError):   # k > 16
            dr.dm.step([30], [gen.chain_tree(1, [])], dr.feat[:1].cuda(), 17)
        with pytest.raises(ValueError):        # features on the host
            dr.dm.step([30], [gen.chain_tree(1, [])], dr.feat[:1], 4)
    finally:
        dr.close()
