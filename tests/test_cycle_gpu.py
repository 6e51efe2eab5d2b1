"""The draft-and-verify cycle on the GPU, through the C ABI, against the fp64
oracle: the target's features of a step's nodes, the draft catching up on
accepted tokens with those features, and whole cycles (draft tree, verify,
accept, commit, features, extend), which must emit exactly the target's
greedy tokens (the paper's losslessness, Sec. 5) whatever the draft.

A draft equal to a one-layer target (TGF passing the token embedding
through, the target's layer, the identity as predict head) must also track
the target: its trees then contain the greedy path, so several drafts are
accepted per cycle, which only happens when the draft's cache and input
features follow the accepted tokens.  Every case prints its name first.
"""

from dataclasses import replace

import numpy as np
import pytest
import torch

from tests import harness as H
import oracle
from oracle import draft as od
from workloads import gen
from workloads.configs import DRAFTS, TINY, DraftShape

pytestmark = pytest.mark.gpu

FEAT_TOL = 1e-3   # of the row's largest |feature| (split-bf16 GEMMs in fp32 vs fp64)
TOKEN_GAP = 2e-3
LOGP_TOL = 2e-3


def say(msg):
    print(f"[gpu-case] {msg}", flush=True)


class Pair:
    """A target verifier (its prefix cache the fp64 prefill of seeded random
    tokens, in bf16) and a draft model of it on the same stream.  draft_kv(b,
    kv) gives the draft layer's prefix (K, V) of sequence b, bf16 torch."""

    def __init__(self, ds, mw, dw, prefixes, draft_kv, max_tree=64, extra=192):
        import paper_2502_11018_amd as P
        m = ds.target
        self.m, self.ds, self.prefixes = m, ds, list(prefixes)
        self.ow = oracle.OracleWeights(mw)
        self.kv = [H.prefix_kv_prefill(self.ow, np.random.default_rng(100 + b).integers(0, m.vocab, p))
                   for b, p in enumerate(prefixes)]
        cap = ((max(prefixes) + extra + 63) // 64) * 64
        say(f"pair {m.name}: prefixes {prefixes} cap {cap}")
        mw_gpu = mw.to("cuda")
        self.v = P.TreeVerifier(m, mw_gpu, max_batch=len(prefixes), max_tree=max_tree, max_depth=max_tree - 1,
                                kv_capacity=cap)
        for b, kv in enumerate(self.kv):
            for l in range(m.n_layers):
                self.v.write_prefix(l, b, torch.from_numpy(kv.K[l]).to(torch.bfloat16).cuda(),
                                    torch.from_numpy(kv.V[l]).to(torch.bfloat16).cuda())
        self.d = P.DraftModel(ds, dw.to("cuda"), mw_gpu, max_batch=len(prefixes), max_tree=max_tree,
                              max_depth=max_tree - 1, kv_capacity=cap)
        self.draft_prefix = []
        for b in range(len(prefixes)):
            k, v = draft_kv(b, self.kv[b])
            self.draft_prefix.append((k.double().numpy(), v.double().numpy()))
            self.d.write_prefix(b, k.cuda(), v.cuda())
        torch.cuda.synchronize()

    def close(self):
        self.d.close()
        self.v.close()


def synthetic_draft_kv(ds):
    return lambda b, kv: gen.synthetic_kv(ds.layer, 0, b, kv.length, 5)


def target_layer0_kv(b, kv):
    return (torch.from_numpy(kv.K[0]).to(torch.bfloat16), torch.from_numpy(kv.V[0]).to(torch.bfloat16))


def self_draft(lm_scale=8.0):
    """A one-layer tiny target (LM head scaled so that its distributions are
    peaked) and a draft equal to it: W_m = [0 | I] and zero biases (h = the
    token embedding), W_d = 0 (o = h), the target's layer, W_p = I."""
    m = replace(TINY, name="tiny-1l", n_layers=1)
    mw = gen.make_weights(m, 0)
    mw.lm_head = (mw.lm_head.float() * lm_scale).to(torch.bfloat16)
    ds = DraftShape(m, tgf_dim=128, k=10, depth=6, n_total=60)
    d, e = m.d_model, ds.tgf_dim
    bf = lambda a: a.to(torch.bfloat16)  # noqa: E731
    eye, zd = torch.eye(d), torch.zeros(d)
    t = {"w_m": bf(torch.cat([torch.zeros(d, d), eye], 1)), "b_m": bf(zd), "ln_h_g": bf(torch.ones(d)),
         "ln_h_b": bf(zd), "ln_x_g": bf(torch.ones(d)), "ln_x_b": bf(zd), "w_u": bf(torch.zeros(e, 2 * d)),
         "b_u": bf(torch.zeros(e)), "w_d": bf(torch.zeros(d, e)), "b_d": bf(zd), "w_p": bf(eye), "b_p": bf(zd),
         "w_r": bf(eye), "b_r": bf(zd)}
    return ds, mw, gen.DraftWeights(ds, t, dict(mw.layers[0]))


def test_target_features_match_oracle():
    """Features (hidden state after the last layer, before the final norm) of
    every node of two trees, and zero rows for -1."""
    ds = DRAFTS["tiny"]
    mw = gen.make_weights(ds.target, 0)
    pr = Pair(ds, mw, gen.make_draft_weights(ds, 3), [37, 90], synthetic_draft_kv(ds))
    try:
        import paper_2502_11018_amd as P
        trees = [gen.random_tree((3, 4, 2), ds.target.vocab, 60 + b)[0] for b in range(2)]
        say("features: before any step")
        with pytest.raises(P.GriffinError):
            pr.v.features([[0]])
        pr.v.step(pr.prefixes, trees)
        n = max(t.n for t in trees) + 1
        nodes = np.full((2, n), -1, dtype=np.int32)
        for b, t in enumerate(trees):
            nodes[b, : t.n] = np.arange(t.n)[::-1]      # any order
        say(f"features: {[t.n for t in trees]} nodes")
        F = pr.v.features(nodes).cpu().numpy()
        for b, t in enumerate(trees):
            ref = oracle.verify_tree(pr.ow, pr.kv[b].fn(), t, pr.prefixes[b]).hidden
            for j in range(n):
                if nodes[b, j] < 0:
                    assert not F[b, j].any()
                    continue
                row = ref[nodes[b, j]]
                err = np.abs(F[b, j] - row).max() / np.abs(row).max()
                assert err < FEAT_TOL, (b, j, err)
        with pytest.raises(P.GriffinError):      # node outside the tree of sequence 0
            pr.v.features([[trees[0].n], [0]])
    finally:
        pr.close()


def test_draft_extend_matches_oracle():
    """Extend the draft's cache by chains of 4 and 2 tokens with given
    features, then run one pass over a new root: its top-k against the
    oracle's pass over the prefix plus the chain's K/V (bf16, as cached)."""
    ds = DRAFTS["tiny"]
    m, k = ds.target, ds.k
    mw = gen.make_weights(m, 0)
    dw = gen.make_draft_weights(ds, 3)
    pr = Pair(ds, mw, dw, [30, 61], synthetic_draft_kv(ds))
    try:
        dow = od.DraftOracleWeights(dw, pr.ow)
        chains = [[11, 250, 3, 77], [500, 8]]
        T, d = pr.d.max_tree, m.d_model
        feats = gen.draft_root_features(d, 2 * T, 21).view(2, T, d).contiguous()
        say(f"extend: chains {[len(c) for c in chains]}")
        pr.d.extend(pr.prefixes, chains, feats.cuda())
        roots = [900, 42]
        root_feat = gen.draft_root_features(d, 2, 23)
        P2 = [p + len(c) for p, c in zip(pr.prefixes, chains)]
        tok, lp = pr.d.step(P2, [gen.chain_tree(r, []) for r in roots], root_feat.cuda(), k)
        compared = 0
        for b, c in enumerate(chains):
            Kp, Vp = pr.draft_prefix[b]
            ch = od.draft_forward(dow, gen.chain_tree(c[0], c[1:]), feats[b, : len(c)].double().numpy(), (Kp, Vp),
                                  pr.prefixes[b])
            K2 = np.concatenate([Kp, H.bf16_round(ch.k).transpose(1, 0, 2)], axis=1)
            V2 = np.concatenate([Vp, H.bf16_round(ch.v).transpose(1, 0, 2)], axis=1)
            r = od.draft_forward(dow, gen.chain_tree(roots[b], []), root_feat[b: b + 1].double().numpy(), (K2, V2),
                                 P2[b])
            otok, olp = od.topk_logprobs(r.logits, k)
            assert np.abs(lp[b, 0] - olp[0]).max() < LOGP_TOL
            srt = np.sort(r.logits[0])[::-1]
            if (-np.diff(srt[: k + 1])).min() > TOKEN_GAP:
                compared += 1
                assert list(tok[b, 0]) == list(otok[0])
        say(f"extend: top-k compared on {compared}/2 roots")
        with pytest.raises(ValueError):           # a chain longer than max_tree (caught by the binding)
            pr.d.extend(pr.prefixes, [[1] * (T + 1), [2]], feats.cuda())
        # the library's own check, called directly: ETREE, nothing enqueued
        import paper_2502_11018_amd._native as N
        from paper_2502_11018_amd.verifier import _i32, _p32
        from ctypes import c_void_p
        tok = np.zeros((2, T), dtype=np.int32)
        rc = N.lib.griffin_draft_extend(pr.d.h, 2, _p32(_i32(P2)), _p32(_i32([T + 1, 1])), _p32(tok),
                                        c_void_p(feats.cuda().data_ptr()))
        assert rc == N.CODES["GRIFFIN_ETREE"]
    finally:
        pr.close()


def _run_cycles(pr, ds, roots, n_tokens, root_features):
    from paper_2502_11018_amd.cycle import SpeculativeCycle
    greedy = []
    for b, r in enumerate(roots):
        g, margins, _ = oracle.greedy_chain(pr.ow, pr.kv[b].decode_cache(pr.m), r, n_tokens + 8)
        assert min(margins) > 1e-3, "pick another seed: a near tie in the greedy chain"
        greedy.append([int(t) for t in g])
    cyc = SpeculativeCycle(pr.v, pr.d, ds.k, ds.depth, ds.n_total)
    cyc.start(pr.prefixes, roots, root_features.cuda())
    out = [[] for _ in roots]
    accepted, cycles = 0, 0
    while min(len(o) for o in out) < n_tokens:
        say(f"{pr.m.name}: cycle {cycles} prefix {cyc.prefix}")
        emitted = cyc.cycle()
        for b, toks in enumerate(emitted):
            out[b] += toks
        accepted += sum(cyc.last_accepted)
        cycles += 1
        assert all(n == ds.n_total + 1 for n in cyc.last_tree_nodes)
    for b in range(len(roots)):
        assert out[b][:n_tokens] == greedy[b][:n_tokens], f"sequence {b} diverged from greedy decoding"
    return accepted / (cycles * len(roots))


def test_cycle_with_a_random_draft_is_lossless():
    ds = DRAFTS["tiny"]
    mw = gen.make_weights(ds.target, 0)
    pr = Pair(ds, mw, gen.make_draft_weights(ds, 3), [40, 75], synthetic_draft_kv(ds))
    try:
        rate = _run_cycles(pr, ds, [6, 17], 30, gen.draft_root_features(ds.target.d_model, 2, 11))
        say(f"random draft: {rate:.2f} drafts accepted per cycle")
    finally:
        pr.close()


def test_cycle_with_a_draft_equal_to_the_target_accepts_its_greedy_path():
    ds, mw, dw = self_draft()
    pr = Pair(ds, mw, dw, [40], target_layer0_kv)
    try:
        rate = _run_cycles(pr, ds, [7], 24, gen.draft_root_features(ds.target.d_model, 1, 11))
        say(f"draft equal to the target: {rate:.2f} drafts accepted per cycle")
        assert rate >= 2.0
    finally:
        pr.close()


# ---- temperature > 0: the drafted tree accepted as a deterministic draft --------

ACCEPT_MARGIN_T = 2e-3  # |u - a| below which the fp64 and device tests may differ (logits differ by rounding)
DRAW_MARGIN_T = 1e-3    # distance of u * sum from a cumulative boundary, as a fraction of the sum
DRAW_TOL_T = 2e-3


def _oracle_tree_logits(pr, b, history, tree):
    """fp64 target logits of the nodes of `tree`, whose root follows the
    cached prefix and `history` (the tokens emitted before the root, starting
    with the first root): one oracle pass over the chain with the tree hung
    below it."""
    m = len(history)
    toks = [int(t) for t in history] + [int(t) for t in tree.tokens]
    par = list(range(-1, m)) + [m + int(p) for p in tree.parents[1:]]
    big = gen.Tree(np.asarray(toks, np.int32), np.asarray(par, np.int32))
    return oracle.verify_tree(pr.ow, pr.kv[b].fn(), big, pr.prefixes[b]).logits[m:]


def _run_sampled_cycles(pr, ds, roots, n_cycles, root_features, T, seed):
    """Cycles at temperature T with seeded uniforms; every cycle's emitted
    tokens against the oracle's walk of the same drafted tree over its own
    fp64 logits, with the same uniforms.  A sequence stops being compared at
    its first accept test within ACCEPT_MARGIN_T of its boundary; a draw
    within DRAW_MARGIN_T of a boundary must be a valid draw within
    DRAW_TOL_T, and the comparison goes on from the device's token."""
    from paper_2502_11018_amd.cycle import SpeculativeCycle
    B = len(roots)
    cyc = SpeculativeCycle(pr.v, pr.d, ds.k, ds.depth, ds.n_total, temperature=T)
    cyc.start(pr.prefixes, roots, root_features.cuda())
    rng = np.random.default_rng(seed)
    hist, cur, live = [[] for _ in roots], [int(r) for r in roots], [True] * B
    compared, accepted, draws_checked = 0, 0, 0
    for c in range(n_cycles):
        shape = (B, pr.v.max_tree)
        ua, uf = rng.random(shape, dtype=np.float32), rng.random(shape, dtype=np.float32)
        say(f"{pr.m.name} T={T}: sampled cycle {c} prefix {cyc.prefix}")
        emitted = cyc.cycle(uniforms=(ua, uf))
        assert all(n == ds.n_total + 1 for n in cyc.last_tree_nodes)
        for b in range(B):
            if not live[b]:
                continue
            t = cyc.last_trees[b]
            tree = gen.Tree(np.asarray(t.tokens, np.int32), np.asarray(t.parents, np.int32))
            tr = []
            r = oracle.accept_sampled(tree, _oracle_tree_logits(pr, b, hist[b], tree), None, ua[b, : tree.n],
                                      uf[b, : tree.n], T, tr)
            if any(e[0] == "accept" and abs(e[1]) <= ACCEPT_MARGIN_T for e in tr):
                live[b] = False
                continue
            L = r.length
            assert emitted[b][:-1] == r.tokens[:-1], (c, b, emitted[b], r.tokens)
            _, margin, rr, cdf = [e for e in tr if e[0] == "draw"][0]
            g = emitted[b][-1]
            if margin > DRAW_MARGIN_T:
                assert g == r.tokens[-1], (c, b, g, r.tokens[-1], margin)
            else:
                lo = cdf[g - 1] if g > 0 else 0.0
                assert lo - DRAW_TOL_T <= rr <= cdf[g] + DRAW_TOL_T, (c, b, g, rr, lo, cdf[g])
                draws_checked += 1
            compared += 1
            accepted += L
            hist[b] += [cur[b]] + r.tokens[:-1]
            cur[b] = g
    say(f"{pr.m.name} T={T}: compared {compared} cycles ({draws_checked} boundary draws), {accepted} drafts accepted")
    return compared, accepted


def test_sampled_cycle_with_a_random_draft_matches_oracle():
    ds = DRAFTS["tiny"]
    mw = gen.make_weights(ds.target, 0)
    pr = Pair(ds, mw, gen.make_draft_weights(ds, 3), [40, 75], synthetic_draft_kv(ds))
    try:
        compared, _ = _run_sampled_cycles(pr, ds, [6, 17], 8, gen.draft_root_features(ds.target.d_model, 2, 11),
                                          1.0, 41)
        assert compared >= 8
    finally:
        pr.close()


@pytest.mark.parametrize("T", [1.0, 0.6])
def test_sampled_cycle_with_a_draft_equal_to_the_target_accepts_paths(T):
    """A draft equal to a one-layer target (LM head scaled so that the
    target's distributions stay peaked at T = 1) proposes the target's likely
    tokens, so sampled cycles accept several drafts each, and every emitted
    token follows the oracle's walk."""
    ds, mw, dw = self_draft(lm_scale=32.0)
    pr = Pair(ds, mw, dw, [40], target_layer0_kv)
    try:
        compared, accepted = _run_sampled_cycles(pr, ds, [7], 8, gen.draft_root_features(ds.target.d_model, 1, 11),
                                                 T, 43)
        assert compared >= 4
        assert accepted >= 1.5 * compared
    finally:
        pr.close()
