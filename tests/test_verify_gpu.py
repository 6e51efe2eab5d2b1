"""Parity of the HIP verify pass with the fp64 oracle, through the C ABI (GPU).

Every case prints its name before touching the GPU so that a failing run
names the case it was in."""

import numpy as np
import pytest
import torch

import oracle
from workloads import gen
from workloads.configs import get_workload
from tests import harness as H

pytestmark = pytest.mark.gpu


def say(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _lib():
    import paper_2502_11018_amd as P
    return P


class Setup:
    """Weights on both sides, prefix caches, oracle results and a verifier."""

    def __init__(self, name, n_trees, max_tree=64, max_depth=None, kv_extra=0, stream=None):
        P = _lib()
        self.w = get_workload(name)
        m = self.w.model
        self.mw = gen.make_weights(m, self.w.weight_seed)
        self.ow = oracle.OracleWeights(self.mw)
        self.dev = torch.device("cuda")
        self.mw_gpu = self.mw.to(self.dev)
        self.max_tree = max_tree
        self.max_depth = max_depth if max_depth is not None else max_tree - 1
        self.cap = ((max(self.w.prefixes()) + max_tree + kv_extra + 63) // 64) * 64
        self.kvs = []
        for b in range(self.w.batch):
            seq_case = H.build_sequence(self.ow, self.w, 0, b)
            self.kvs.append(seq_case.kv)
        self.cases = [[H.build_sequence(self.ow, self.w, i, b, kv=self.kvs[b]) for b in range(self.w.batch)]
                      for i in range(n_trees)]
        say(f"{name}: init verifier cap={self.cap} max_tree={max_tree}")
        self.v = P.TreeVerifier(m, self.mw_gpu, max_batch=self.w.batch, max_tree=max_tree,
                                max_depth=self.max_depth, kv_capacity=self.cap, stream=stream)
        for b, kv in enumerate(self.kvs):
            for l in range(m.n_layers):
                self.v.write_prefix(l, b, torch.from_numpy(kv.K[l]).to(torch.bfloat16).to(self.dev),
                                    torch.from_numpy(kv.V[l]).to(torch.bfloat16).to(self.dev))
        torch.cuda.synchronize()

    def run(self, trees, prefix=None, logits=True):
        B = len(trees)
        prefix = self.w.prefixes()[:B] if prefix is None else prefix
        out = torch.full((B * self.max_tree, self.w.model.vocab), float("nan"), device=self.dev) if logits else None
        self.v.step(prefix, trees, out)
        acc = self.v.accept(check=False)
        pred = self.v.predictions()
        lg = out.view(B, self.max_tree, -1).cpu().numpy() if logits else None
        return lg, pred, acc


@pytest.fixture(scope="module")
def tiny():
    s = Setup("tiny", n_trees=16)
    yield s
    s.v.close()


def test_tiny_all_trees_match_oracle(tiny):
    stats = []
    for i, cases in enumerate(tiny.cases):
        say(f"tiny tree {i}")
        c = cases[0]
        os_ = H.oracle_sequence(tiny.ow, c)
        lg, pred, acc = tiny.run([c.tree])
        assert acc.status == 0
        st = H.check_parity(os_, lg[0, : c.tree.n], pred[0, : c.tree.n], acc.sequence(0))
        # the device's top-2 margin: exact for its own logits, within twice their error of the oracle's
        mg = tiny.v.margins()[0]
        own = np.sort(lg[0, : c.tree.n].astype(np.float64), axis=1)
        assert np.allclose(mg[: c.tree.n], own[:, -1] - own[:, -2], rtol=0, atol=1e-6)
        err = np.abs(lg[0, : c.tree.n] - os_.logits).max(axis=1)
        assert np.all(np.abs(mg[: c.tree.n] - os_.margin) <= 2 * err + 1e-7)
        assert np.all(mg[c.tree.n:] == -1)
        # planted root-to-leaf greedy paths are accepted in full
        assert int(acc.length[0]) >= len(c.plant_path) or not st["accept_checked"]
        stats.append(st)
    say(f"tiny stats: max rel err {max(s['max_rel'] for s in stats):.2e}, "
        f"accept checked {sum(s['accept_checked'] for s in stats)}/16, "
        f"lengths {[s['L'] for s in stats]}")
    # trees whose accepted nodes all have a top-2 margin above the gate are
    # compared bit-exactly; with logit std ~0.3 (d = 256) about a third qualify
    assert sum(s["accept_checked"] for s in stats) >= 3


@pytest.mark.parametrize("name", ["small-gqa", "small-mha", "small-moe", "small-chain2"])
def test_small_workloads_match_oracle(name):
    """small-chain2 is a ragged serving batch: 16 sequences with prefixes of
    20..200 tokens and chains of 0..2 drafts in 3-row slots."""
    s = Setup(name, n_trees=3, max_tree=get_workload(name).max_tree)
    try:
        checked = 0
        for i, cases in enumerate(s.cases):
            say(f"{name} step {i} batch {len(cases)}")
            lg, pred, acc = s.run([c.tree for c in cases])
            moe = s.w.model.n_experts > 1
            rl = s.v.router_logits() if moe else None       # [L, B, max_tree, E]
            for b, c in enumerate(cases):
                os_ = H.oracle_sequence(s.ow, c)
                excl = set()
                if moe:
                    err, gap, excl, near = H.router_check(os_, rl[:, b], s.w.model.top_k)
                    say(f"{name} step {i} seq {b}: router logit error {err:.2e}, gap {gap:.2e}, "
                        f"nodes with other experts on their path {len(excl)}, with a near tie {len(near)}")
                    # at this size the gap is the 1e-4 floor and no routing is that close
                    assert not excl and not near
                st = H.check_parity(os_, lg[b, : c.tree.n], pred[b, : c.tree.n], acc.sequence(b), excl)
                checked += st["accept_checked"]
                if st["accept_checked"]:
                    assert int(acc.length[b]) >= len(c.plant_path)
        assert checked >= 1
    finally:
        s.v.close()


def test_hand_trees(tiny):
    m = tiny.w.model
    kv = tiny.kvs[0]
    ow = tiny.ow
    r = np.random.default_rng(5)
    trees = {
        "one_node": gen.chain_tree(17, []),
        "chain6": gen.chain_tree(3, list(r.integers(0, m.vocab, 6))),
        "star64": gen.Tree(r.integers(0, m.vocab, 64).astype(np.int32),
                           np.array([-1] + [0] * 63, dtype=np.int32)),
        "dup_siblings": gen.Tree(np.array([5, 9, 9, 9, 4, 4], dtype=np.int32),
                                 np.array([-1, 0, 0, 0, 1, 2], dtype=np.int32)),
    }
    greedy, _, _ = oracle.greedy_chain(ow, kv.decode_cache(m), 3, 7)
    trees["chain_greedy"] = gen.chain_tree(3, greedy[:6])
    for name, t in trees.items():
        say(f"hand tree {name}")
        c = H.SeqCase(None, kv, t, [], [], [])
        os_ = H.oracle_sequence(ow, c)
        lg, pred, acc = tiny.run([t])
        H.check_parity(os_, lg[0, : t.n], pred[0, : t.n], acc.sequence(0))
        if name == "dup_siblings":
            # identical contexts: equal up to the summation order of the masked slots
            for i, j in ((1, 2), (4, 5)):
                assert np.abs(lg[0, i] - lg[0, j]).max() < 1e-3 * np.abs(lg[0, i]).max()
    # the greedy chain is accepted in full (6 draft tokens + the next greedy token)
    lg, pred, acc = tiny.run([trees["chain_greedy"]])
    L, toks, _ = acc.sequence(0)
    assert L == 6 and toks == greedy[:7]


def test_chain_tree_equals_sequential_decoding_on_gpu(tiny):
    # logits of node k of a chain equal one-node verifies after committing the chain prefix
    m = tiny.w.model
    toks = [3, 41, 7, 600, 12]
    chain = gen.chain_tree(9, toks)
    say("chain vs sequential")
    lg, _, _ = tiny.run([chain])
    P = tiny.w.prefix_len
    seq = [9] + toks
    for k in range(len(seq)):
        # nodes 0..k-1 of the chain are already in the cache at slots P..P+k-1
        # from the chain step above; verify token k alone at prefix P+k
        lg1, _, _ = tiny.run([gen.chain_tree(seq[k], [])], prefix=[P + k])
        rel = np.abs(lg1[0, 0] - lg[0, k]).max() / (lg[0, k].max() - lg[0, k].min())
        assert rel < 1e-2, (k, rel)
        # restore the chain's slots for the next k (the 1-node step overwrote slot P+k)
        tiny.run([chain], logits=False)


def test_prefix_zero_and_accept_walk_golden():
    P = _lib()
    from tests.test_oracle_golden import ACCEPT_CASES
    trees = [gen.Tree(np.array(c["tokens"], dtype=np.int32), np.array(c["parents"], dtype=np.int32))
             for c in ACCEPT_CASES]
    max_tree = 8
    pred = np.zeros((len(trees), max_tree), dtype=np.int32)
    for b, c in enumerate(ACCEPT_CASES):
        pred[b, : len(c["pred"])] = c["pred"]
    say("accept walk golden")
    res = P.accept_walk(trees, pred, max_tree=max_tree, max_depth=7, vocab=100)
    for b, c in enumerate(ACCEPT_CASES):
        L, toks, path = res.sequence(b)
        assert (L, toks, path) == (c["L"], c["accepted"], c["path"]), c["name"]
        assert list(res.tokens[b, L + 1:]) == [-1] * (7 - L)
        assert list(res.path[b, L:]) == [-1] * (7 - L)


def test_empty_prefix_matches_oracle():
    P = _lib()
    w = get_workload("small-gqa")
    m = w.model
    mw = gen.make_weights(m, 0)
    ow = oracle.OracleWeights(mw)
    empty = H.PrefixKV([np.zeros((m.n_kv_heads, 0, m.head_dim))] * m.n_layers,
                       [np.zeros((m.n_kv_heads, 0, m.head_dim))] * m.n_layers)
    tree, _ = gen.random_tree((3, 4, 4), m.vocab, 11)
    os_ = H.oracle_sequence(ow, H.SeqCase(None, empty, tree, [], [], []))
    say("empty prefix")
    with P.TreeVerifier(m, mw.to("cuda"), max_batch=1, max_tree=16, max_depth=15, kv_capacity=64) as v:
        out = torch.empty((16, m.vocab), device="cuda")
        v.step([0], [tree], out)
        acc = v.accept()
        H.check_parity(os_, out[: tree.n].cpu().numpy(), v.predictions()[0], acc.sequence(0))


def test_scores_past_the_attention_cap_match_oracle():
    """Prefix keys after the first 32 are scaled by 2^14, so inside the first
    key split (two 32-key blocks: 1024 keys over 16 splits) the second block's
    scores exceed the first block's maximum by thousands of log2 units, far
    past the 2^64 bound the attention kernel allows its unnormalised
    probabilities (they overflow to inf there).  That split is flagged and
    the merge recomputes it exactly, ignoring its overflowed partial; the
    rest of the pass is unchanged.  The softmax then concentrates on a few keys, on both
    sides."""
    P = _lib()
    w = get_workload("small-gqa")
    m = w.model
    mw = gen.make_weights(m, 0)
    ow = oracle.OracleWeights(mw)
    plen = 1024
    K, V = [], []
    for l in range(m.n_layers):
        k, v = gen.synthetic_kv(m, l, 0, plen, 7, "cpu")
        k = k.to(torch.float32)
        k[:, 32:, :] *= 16384.0  # a power of two: still exactly bf16
        K.append(k.to(torch.float64).numpy())
        V.append(v.to(torch.float64).numpy())
    tree, _ = gen.random_tree((3, 4, 4), m.vocab, 5)
    os_ = H.oracle_sequence(ow, H.SeqCase(None, H.PrefixKV(K, V), tree, [], [], []))
    say("scores past the attention cap")
    with P.TreeVerifier(m, mw.to("cuda"), max_batch=1, max_tree=16, max_depth=15, kv_capacity=plen + 64) as v:
        for l in range(m.n_layers):
            v.write_prefix(l, 0, torch.from_numpy(K[l]).to(torch.bfloat16).cuda(),
                           torch.from_numpy(V[l]).to(torch.bfloat16).cuda())
        out = torch.empty((16, m.vocab), device="cuda")
        v.step([plen], [tree], out)
        acc = v.accept()
        # the merge recomputes the flagged splits from the bf16 cache: a larger, bounded error
        st = H.check_parity(os_, out[: tree.n].cpu().numpy(), v.predictions()[0], acc.sequence(0),
                            regress_tol=5e-3)
    say(f"scores past the attention cap: max rel err {st['max_rel']:.2e}")


def test_errors_leave_cache_untouched(tiny):
    P = _lib()
    v = tiny.v
    k0, v0 = v.k_cache.clone(), v.v_cache.clone()
    good = tiny.cases[0][0].tree
    bad_parent = good.copy()
    bad_parent.parents[3] = 7
    bad_token = good.copy()
    bad_token.tokens[2] = tiny.w.model.vocab
    cases = [([tiny.w.prefix_len], [bad_parent], "GRIFFIN_ETREE"),
             ([tiny.w.prefix_len], [bad_token], "GRIFFIN_ETOKEN"),
             ([tiny.cap - 3], [good], "GRIFFIN_ECAPACITY")]
    for prefix, trees, code in cases:
        say(f"error path {code}")
        with pytest.raises(P.GriffinError) as ei:
            v.step(prefix, trees)
        assert ei.value.name == code
    torch.cuda.synchronize()
    assert torch.equal(v.k_cache, k0) and torch.equal(v.v_cache, v0)


def test_accept_before_step_is_an_order_error():
    P = _lib()
    w = get_workload("tiny")
    mw = gen.make_weights(w.model, 0).to("cuda")
    say("EORDER")
    with P.TreeVerifier(w.model, mw, max_batch=1, max_tree=16, max_depth=4, kv_capacity=192) as v:
        with pytest.raises(P.GriffinError) as ei:
            v.accept()
        assert ei.value.name == "GRIFFIN_EORDER"


def test_bitwise_deterministic(tiny):
    t = tiny.cases[1][0].tree
    say("determinism")
    a, pa, _ = tiny.run([t])
    b, pb, _ = tiny.run([t])
    assert np.array_equal(a[0, : t.n].view(np.uint32), b[0, : t.n].view(np.uint32))
    assert np.array_equal(pa, pb)


def test_batched_equals_separate():
    name = "small-mha"
    s = Setup(name, n_trees=1)
    try:
        trees = [c.tree for c in s.cases[0]]
        say(f"{name} batched vs separate")
        lg, pred, acc = s.run(trees)
        for b, t in enumerate(trees):
            # one sequence at a time in row b (other rows absent) must give the same bits
            single = [gen.chain_tree(0, []) for _ in trees]
            single[b] = t
            lg1, pred1, acc1 = s.run(single)
            assert np.array_equal(lg[b, : t.n].view(np.uint32), lg1[b, : t.n].view(np.uint32))
            assert acc.sequence(b) == acc1.sequence(b)
    finally:
        s.v.close()


def test_gpu_prefill_by_chain_steps_matches_oracle_prefill():
    # build the prefix cache on the GPU by verifying chains and committing
    # them (prefix += n), then compare with the oracle's fp64 prefill
    P = _lib()
    w = get_workload("tiny")
    m = w.model
    mw = gen.make_weights(m, 0)
    ow = oracle.OracleWeights(mw)
    toks = gen.prefix_tokens(w)
    kv = H.prefix_kv_prefill(ow, toks)
    say("gpu chain prefill")
    with P.TreeVerifier(m, mw.to("cuda"), max_batch=1, max_tree=32, max_depth=31, kv_capacity=192) as v:
        p = 0
        while p < len(toks):
            chunk = [int(t) for t in toks[p: p + 32]]
            v.step([p], [gen.chain_tree(chunk[0], chunk[1:])])
            v.accept()
            p += len(chunk)
        torch.cuda.synchronize()
        for l in range(m.n_layers):
            kg = v.k_cache[l, 0, :, : len(toks), :].float().cpu().numpy()
            vg = v.read_v(l, 0, len(toks)).float().cpu().numpy()
            for ref, got in ((kv.K[l], kg), (kv.V[l], vg)):
                rel = np.abs(got - ref).max() / np.abs(ref).max()
                assert rel < 3e-2, (l, rel)


def test_graph_replay_matches_plain_launches():
    """Steps replayed from captured HIP graphs give the same bits as plain
    launches, on every replay, with plain steps and synchronisations between
    the replays and several graph keys in use: two batch sizes, and prefix
    lengths that change the key-split plan (one full prefix beside a short
    one: the same merge slot count as equal prefixes, with another split
    table) or the merge's slot count itself (all prefixes short: one split
    each, one slot instead of four), so a new graph."""
    name = "small-gqa"
    # a stream of its own: the library captures and replays graphs only on a
    # non-default stream
    s = Setup(name, n_trees=3, stream=torch.cuda.Stream())
    try:
        m = s.w.model
        B = s.w.batch
        trees = [[c.tree for c in s.cases[i]] for i in range(3)]
        out = torch.empty((B * s.max_tree, m.vocab), device=s.dev)

        other = {"uneven": [s.w.prefix_len] + [40] * (B - 1), "short": [40] * B}
        # a step writes its tree's K/V at slots prefix + i: a short step
        # overwrites prefix slots that the full-prefix steps read, so the
        # cache is restored after it
        torch.cuda.synchronize()
        kc0, vc0 = s.v.k_cache.clone(), s.v.v_cache.clone()

        def step(ts, prefixes=None):
            out.fill_(float("nan"))
            s.v.step(prefixes or [s.w.prefix_len] * len(ts), ts, out)
            acc = s.v.accept(check=False)
            res = out[: len(ts) * s.max_tree].cpu().numpy().copy(), s.v.predictions(), \
                [acc.sequence(b) for b in range(len(ts))]
            if prefixes is not None:
                torch.cuda.synchronize()
                s.v.k_cache.copy_(kc0)
                s.v.v_cache.copy_(vc0)
                torch.cuda.synchronize()
            return res

        say(f"{name}: plain launches")
        s.v.set_graphs(False)
        ref = [step(t) for t in trees]
        ref1 = step(trees[0][:1])
        ref_o = {k: step(trees[0], pl) for k, pl in other.items()}
        s.v.set_graphs(True)
        for rep in range(3):
            for i, t in enumerate(trees):
                say(f"{name}: graph replay {rep} tree set {i}")
                lg, pred, acc = step(t)
                assert np.array_equal(lg.view(np.uint32), ref[i][0].view(np.uint32))
                assert np.array_equal(pred, ref[i][1]) and acc == ref[i][2]
                if i == 0:  # the other prefix patterns between the equal ones
                    for k, pl in other.items():
                        lg, pred, acc = step(t, pl)
                        assert np.array_equal(lg.view(np.uint32), ref_o[k][0].view(np.uint32)), k
                        assert np.array_equal(pred, ref_o[k][1]) and acc == ref_o[k][2], k
            lg1, pred1, acc1 = step(trees[0][:1])  # batch 1: a second graph
            assert np.array_equal(lg1.view(np.uint32), ref1[0].view(np.uint32)) and acc1 == ref1[2]
            s.v.set_graphs(False)            # plain step between replays
            step(trees[(rep + 1) % 3])
            torch.cuda.synchronize()
            s.v.set_graphs(True)
    finally:
        s.v.close()


@pytest.mark.parametrize("name", ["tiny", "small-gqa"])
def test_speculative_loop_is_lossless(name):
    """The paper's decoding is lossless (Sec. 5): cycles of step / accept /
    commit on random draft trees, part of each tree planted with the target's
    true continuation, emit exactly the oracle's greedy tokens; every
    sequence of a batch runs its own loop at its own prefix length."""
    N = 40
    s = Setup(name, n_trees=1, kv_extra=N + 8)
    try:
        m = s.w.model
        B = s.w.batch
        rng = np.random.default_rng(5)
        greedy, roots = [], []
        for b in range(B):
            root = int(s.cases[0][b].tree.tokens[0])
            g, margins, _ = oracle.greedy_chain(s.ow, s.kvs[b].decode_cache(m), root, N + 8)
            assert min(margins) > 1e-3, "pick another seed: a near tie in the greedy chain"
            greedy.append([int(t) for t in g])
            roots.append(root)
        P = [s.w.prefix_len] * B
        out = [[] for _ in range(B)]
        cycle, accepted = 0, 0
        while min(len(o) for o in out) < N:
            trees = []
            for b in range(B):
                tree, _ = gen.random_tree(s.w.widths, m.vocab, 9000 + 97 * cycle + b)
                tree.tokens[0] = roots[b]
                depth = tree.depths()
                deepest = [i for i in range(1, tree.n) if depth[i] == depth.max()]
                path = tree.root_path(deepest[int(rng.integers(len(deepest)))])
                l = int(rng.integers(0, len(path) + 1))
                trees.append(gen.apply_plant(tree, path[:l], greedy[b][len(out[b]): len(out[b]) + l]))
            say(f"{name}: cycle {cycle} prefix {P}")
            s.v.step(P, trees)
            acc = s.v.accept()
            s.v.commit()
            for b in range(B):
                L, toks, _ = acc.sequence(b)
                out[b] += toks
                P[b] += L + 1
                roots[b] = toks[-1]
                accepted += L
            cycle += 1
        for b in range(B):
            assert out[b][:N] == greedy[b][:N], f"sequence {b} diverged from greedy decoding"
        assert accepted > cycle  # the planted parts were accepted (more than one token per cycle on average)
    finally:
        s.v.close()


def test_activation_precision_switch_drops_stale_graphs(tiny):
    """Switching the GEMM activations to bf16 alone changes the logits (a
    different kernel variant runs, not a stale graph), and switching back
    gives the default's bits again, with graph replay on throughout."""
    m = tiny.w.model
    trees = [tiny.cases[0][0].tree]
    out = torch.empty((tiny.max_tree, m.vocab), device=tiny.dev)

    def logits():
        out.fill_(float("nan"))
        tiny.v.step([tiny.w.prefix_len], trees, out)
        tiny.v.accept(check=False)
        return out[: trees[0].n].cpu().numpy().copy()

    say("tiny: activation precision switch")
    ref = logits()
    assert np.array_equal(logits(), ref)            # graph replay of the default
    try:
        tiny.v.set_bf16_activations(True)
        alt = logits()
        assert np.isfinite(alt).all() and not np.array_equal(alt, ref)
        assert np.array_equal(logits(), alt)        # its own graph replays the same bits
    finally:
        tiny.v.set_bf16_activations(False)
    assert np.array_equal(logits(), ref)


def test_nan_in_the_lm_head_is_reported(tiny):
    """A NaN in one row of the LM head makes that vocabulary entry NaN at every
    node: griffin_accept reports GRIFFIN_ENUMERIC and still writes its
    outputs, which are the walk over the argmax of the remaining entries."""
    P = _lib()
    m = tiny.w.model
    c = tiny.cases[0][0]
    os_ = H.oracle_sequence(tiny.ow, c)
    bad = int(os_.pred[0])          # the root's own argmax, so the NaN hides the winner there
    lm = tiny.mw.lm_head.clone()
    lm[bad, 7] = float("nan")
    w_nan = gen.ModelWeights(m, tiny.mw.embed, lm, tiny.mw.final_norm, tiny.mw.layers).to("cuda")
    say("tiny: NaN in one LM-head row")
    with P.TreeVerifier(m, w_nan, max_batch=1, max_tree=tiny.max_tree, max_depth=tiny.max_depth,
                        kv_capacity=tiny.cap) as v:
        for l in range(m.n_layers):
            v.write_prefix(l, 0, torch.from_numpy(c.kv.K[l]).to(torch.bfloat16).cuda(),
                           torch.from_numpy(c.kv.V[l]).to(torch.bfloat16).cuda())
        out = torch.empty((tiny.max_tree, m.vocab), device="cuda")
        v.step([tiny.w.prefix_len], [c.tree], out)
        with pytest.raises(P.GriffinError) as ei:
            v.accept()
        assert ei.value.name == "GRIFFIN_ENUMERIC"
        acc = v.accept(check=False)
        assert P.STATUS[acc.status] == "GRIFFIN_ENUMERIC"
        lg = out[: c.tree.n].cpu().numpy()
        pred = v.predictions()[0][: c.tree.n]
    assert np.isnan(lg[:, bad]).all()
    # the argmax skips the NaN entry: the oracle's argmax with that entry removed
    ol = os_.logits.copy()
    ol[:, bad] = -np.inf
    srt = np.sort(ol, axis=1)
    for i in range(c.tree.n):
        if srt[i, -1] - srt[i, -2] > H.MARGIN_GATE:
            assert pred[i] == int(np.argmax(ol[i])), i
    assert pred[0] != bad
    own = oracle.accept_dfs(c.tree, pred)
    assert acc.sequence(0) == (own.length, own.tokens, own.path)
