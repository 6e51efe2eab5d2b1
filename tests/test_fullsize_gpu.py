"""Full-size parity: the verify pass at the benchmark's shapes against the fp64
oracle on the host (GPU).

The weights are generated on the GPU by the seeded generator and copied to the
host for the oracle (the generator is bit-identical on both devices; see
test_generator_is_device_independent).  The prefix KV cache is the workload's
seeded synthetic cache.  Trees come from the workload's pool; a planted tree
carries the oracle's own greedy continuation.  Each case prints its name
before touching the GPU.
"""

import os
import time

import numpy as np
import pytest
import torch

import oracle
from workloads import gen
from workloads.configs import get_workload
from tests import harness as H

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def say(msg):
    print(f"[gpu-case] {msg}", flush=True)


def test_generator_is_device_independent():
    say("generator cpu vs gpu")
    for n, seed, stream, std in [(1 << 20, 0, 7, 0.02), (3 * (1 << 20) + 5, 3, 1 << 20, 1.28)]:
        a = gen.hashed_normal_bf16(n, seed, stream, std, "cpu")
        b = gen.hashed_normal_bf16(n, seed, stream, std, "cuda").cpu()
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))


class LoudKV(H.PrefixKV):
    """PrefixKV that reports the oracle's progress (it reads layer l's cache
    when it reaches layer l), so that a long host computation is never silent."""

    def fn(self):
        t0 = time.time()

        def get(l):
            if l % 8 == 0:
                say(f"  oracle at layer {l} ({time.time() - t0:.0f}s)")
            return self.K[l], self.V[l]
        return get


def _planted(w, ow, kv, max_index=64):
    """First tree of the pool that the workload plants, with its oracle greedy path."""
    for i in range(max_index):
        tree, path = gen.workload_tree(w, i)
        if len(path) >= 3:
            greedy, margins, _ = oracle.greedy_chain(ow, kv.decode_cache(w.model), int(tree.tokens[0]), len(path))
            return i, gen.apply_plant(tree, path, greedy), path, greedy
    raise AssertionError("no planted tree in the pool")


@pytest.mark.parametrize("name", ["llama3-8b", "llama2-7b"])
def test_full_size_verify_matches_oracle(name):
    _full_size_verify(name, bf16_activations=False)


def test_full_size_bf16_activations_error_bound():
    """The opt-in mode with GEMM activations rounded to bf16 (a plain bf16
    forward pass, the paper's setting) instead of bf16 hi + lo.  It does not
    meet the acceptance gate: over 32 layers the logits drift by ~2e-2 of the
    row range and the argmax flips at nodes whose oracle margin is several
    times 1e-2.  Measured here, with a bound on the drift, so that the
    default's need for the low parts stays documented."""
    _full_size_verify("llama3-8b", bf16_activations=True)


def _full_size_verify(name, bf16_activations):
    import paper_2502_11018_amd as P
    w = get_workload(name)
    m = w.model
    t0 = time.time()
    say(f"{name}: generate weights on the GPU (bf16 activations: {bf16_activations})")
    mw_gpu = gen.make_weights(m, w.weight_seed, device="cuda")
    v = P.TreeVerifier(m, mw_gpu, max_batch=1, max_tree=64, max_depth=w.depth, kv_capacity=w.kv_capacity())
    v.set_bf16_activations(bf16_activations)
    Ks, Vs = [], []
    for l in range(m.n_layers):
        k, vv = gen.synthetic_kv(m, l, 0, w.prefix_len, w.weight_seed, "cuda")
        v.write_prefix(l, 0, k, vv)
        Ks.append(k.to(torch.float64).cpu().numpy())
        Vs.append(vv.to(torch.float64).cpu().numpy())
    kv = H.PrefixKV(Ks, Vs)
    say(f"{name}: host copy of the weights for the oracle ({time.time() - t0:.0f}s)")
    ow = oracle.OracleWeights(mw_gpu.to("cpu"), cache=True)
    unplanted = next(gen.workload_tree(w, i)[0] for i in range(64) if not gen.workload_tree(w, i)[1])
    say(f"{name}: oracle greedy continuation ({time.time() - t0:.0f}s)")
    idx, planted, path, greedy = _planted(w, ow, kv)
    for label, tree in (("unplanted", unplanted), (f"planted#{idx}", planted)):
        say(f"{name}: GPU verify {label}")
        logits = torch.empty((64, m.vocab), device="cuda")
        v.step([w.prefix_len], [tree], logits)
        acc = v.accept()
        pred = v.predictions()[0]
        lg = logits[: tree.n].cpu().numpy()
        say(f"{name}: oracle verify {label} ({time.time() - t0:.0f}s)")
        os_ = H.oracle_sequence(ow, H.SeqCase(None, kv, tree, [], [], []))
        if bf16_activations:
            span = os_.logits.max(axis=1) - os_.logits.min(axis=1)
            drift = (np.abs(lg - os_.logits).max(axis=1) / span).max()
            gated = [i for i in range(tree.n) if os_.margin[i] > 1e-2]
            flips = [i for i in gated if pred[i] != np.argmax(os_.logits[i])]
            say(f"{name} {label} (bf16 activations): logit drift {drift:.2e} of the range, argmax flips at "
                f"{len(flips)}/{len(gated)} gated nodes (largest margin {max([os_.margin[i] for i in flips], default=0):.3f})")
            assert drift < 5e-2
            continue
        st = H.check_parity(os_, lg, pred[: tree.n], acc.sequence(0))
        rel = np.abs(lg - os_.logits).max(axis=1)
        say(f"{name} {label}: max rel err {st['max_rel']:.2e}, max abs err {rel.max():.3e}, "
            f"gated {st['gated']}/{st['total']}, accept checked {st['accept_checked']}, L={st['L']}")
        if label.startswith("planted") and st["accept_checked"]:
            assert int(acc.length[0]) >= len(path)
    v.close()


def test_full_size_moe_verify_matches_oracle():
    """Mixtral-8x7B shape (about 94 GB of bf16 weights, 8 experts, top-2): one
    unplanted tree through all 32 layers.  The device's router logits are
    compared with the oracle's; nodes whose root path chose other experts
    than the oracle (each such choice must be a near tie within the measured
    router-logit error) are left out of the gates and counted."""
    import paper_2502_11018_amd as P
    w = get_workload("mixtral-8x7b")
    m = w.model
    t0 = time.time()
    say("mixtral-8x7b: generate weights on the GPU")
    mw_gpu = gen.make_weights(m, w.weight_seed, device="cuda")
    v = P.TreeVerifier(m, mw_gpu, max_batch=1, max_tree=64, max_depth=w.depth, kv_capacity=w.kv_capacity())
    Ks, Vs = [], []
    for l in range(m.n_layers):
        k, vv = gen.synthetic_kv(m, l, 0, w.prefix_len, w.weight_seed, "cuda")
        v.write_prefix(l, 0, k, vv)
        Ks.append(k.to(torch.float64).cpu().numpy())
        Vs.append(vv.to(torch.float64).cpu().numpy())
    kv = LoudKV(Ks, Vs)
    tree = next(gen.workload_tree(w, i)[0] for i in range(64) if not gen.workload_tree(w, i)[1])
    say("mixtral-8x7b: GPU verify")
    logits = torch.empty((64, m.vocab), device="cuda")
    v.step([w.prefix_len], [tree], logits)
    acc = v.accept()
    pred = v.predictions()[0]
    lg = logits[: tree.n].cpu().numpy()
    rl = v.router_logits()[:, 0]
    v.close()
    say(f"mixtral-8x7b: host copy of the weights ({time.time() - t0:.0f}s)")
    ow = oracle.OracleWeights(mw_gpu.to("cpu"), cache=False)
    del mw_gpu
    say(f"mixtral-8x7b: oracle verify ({time.time() - t0:.0f}s)")
    os_ = H.oracle_sequence(ow, H.SeqCase(None, kv, tree, [], [], []))
    err, gap, ex, near = H.router_check(os_, rl, m.top_k)
    st = H.check_parity(os_, lg, pred[: tree.n], acc.sequence(0), exclude=ex)
    say(f"mixtral-8x7b: max rel err {st['max_rel']:.2e}, gated {st['gated']}/{st['total']}, "
        f"router logit error {err:.2e}, near-tie gap {gap:.2e}, nodes with other experts on their path "
        f"{len(ex)} (with a near tie: {len(near)}), accept checked {st['accept_checked']} ({time.time() - t0:.0f}s)")
    # the MoE path is checked on almost every node, not on the few a wide gap leaves
    assert len(ex) <= tree.n // 10


def test_full_size_long_context_batch_matches_oracle():
    """Llama-3-8B shape, batch 8 x 16384-token prefixes (about 17 GB of KV),
    eight different trees packed into one verify call; sequences 0, 3 and 7
    are checked against the oracle."""
    import paper_2502_11018_amd as P
    w = get_workload("llama3-8b-longctx")
    m = w.model
    B = w.batch
    t0 = time.time()
    say("llama3-8b-longctx: generate weights on the GPU")
    mw_gpu = gen.make_weights(m, w.weight_seed, device="cuda")
    v = P.TreeVerifier(m, mw_gpu, max_batch=B, max_tree=64, max_depth=w.depth, kv_capacity=w.kv_capacity())
    checked = (0, 3, 7)
    host_kv = {b: ([], []) for b in checked}
    for l in range(m.n_layers):
        for b in range(B):
            k, vv = gen.synthetic_kv(m, l, b, w.prefix_len, w.weight_seed, "cuda")
            v.write_prefix(l, b, k, vv)
            if b in checked:
                host_kv[b][0].append(k.to(torch.float64).cpu().numpy())
                host_kv[b][1].append(vv.to(torch.float64).cpu().numpy())
    trees = [gen.workload_tree(w, 0, b)[0] for b in range(B)]
    say(f"llama3-8b-longctx: GPU verify of {B} trees ({time.time() - t0:.0f}s)")
    logits = torch.empty((B * 64, m.vocab), device="cuda")
    v.step([w.prefix_len] * B, trees, logits)
    acc = v.accept()
    pred = v.predictions()
    lg_all = logits.view(B, 64, m.vocab)
    say(f"llama3-8b-longctx: host copy of the weights ({time.time() - t0:.0f}s)")
    ow = oracle.OracleWeights(mw_gpu.to("cpu"), cache=True)
    for b in checked:
        say(f"llama3-8b-longctx: oracle verify of sequence {b} ({time.time() - t0:.0f}s)")
        kv = LoudKV(*host_kv[b])
        os_ = H.oracle_sequence(ow, H.SeqCase(None, kv, trees[b], [], [], []))
        lg = lg_all[b, : trees[b].n].cpu().numpy()
        st = H.check_parity(os_, lg, pred[b, : trees[b].n], acc.sequence(b))
        say(f"llama3-8b-longctx seq {b}: max rel err {st['max_rel']:.2e}, gated {st['gated']}/{st['total']}, "
            f"accept checked {st['accept_checked']}, L={st['L']}")
    v.close()


def test_full_size_ragged_chain2_batch_matches_oracle():
    """Llama-3-8B shape, a serving batch of 16 sequences with prefixes spread
    over 256..2048 tokens and a chain of 2 drafts each, in 3-row slots (48
    node rows in one call); sequences 0, 7 and 15 are checked against the
    oracle."""
    import paper_2502_11018_amd as P
    w = get_workload("llama3-8b-chain2-b16")
    m = w.model
    B, prefix = w.batch, w.prefixes()
    t0 = time.time()
    say(f"llama3-8b-chain2-b16: generate weights on the GPU (prefixes {prefix})")
    mw_gpu = gen.make_weights(m, w.weight_seed, device="cuda")
    v = P.TreeVerifier(m, mw_gpu, max_batch=B, max_tree=w.max_tree, max_depth=w.depth,
                       kv_capacity=w.kv_capacity())
    checked = (0, 7, 15)
    host_kv = {b: ([], []) for b in checked}
    for l in range(m.n_layers):
        for b in range(B):
            k, vv = gen.synthetic_kv(m, l, b, prefix[b], w.weight_seed, "cuda")
            v.write_prefix(l, b, k, vv)
            if b in checked:
                host_kv[b][0].append(k.to(torch.float64).cpu().numpy())
                host_kv[b][1].append(vv.to(torch.float64).cpu().numpy())
    trees = [gen.workload_tree(w, 0, b)[0] for b in range(B)]
    say(f"llama3-8b-chain2-b16: GPU verify of {B} chains ({time.time() - t0:.0f}s)")
    logits = torch.empty((B * w.max_tree, m.vocab), device="cuda")
    v.step(prefix, trees, logits)
    acc = v.accept()
    pred = v.predictions()
    lg_all = logits.view(B, w.max_tree, m.vocab)
    say(f"llama3-8b-chain2-b16: host copy of the weights ({time.time() - t0:.0f}s)")
    ow = oracle.OracleWeights(mw_gpu.to("cpu"), cache=True)
    for b in checked:
        say(f"llama3-8b-chain2-b16: oracle verify of sequence {b}, prefix {prefix[b]} ({time.time() - t0:.0f}s)")
        kv = LoudKV(*host_kv[b])
        os_ = H.oracle_sequence(ow, H.SeqCase(None, kv, trees[b], [], [], []))
        lg = lg_all[b, : trees[b].n].cpu().numpy()
        st = H.check_parity(os_, lg, pred[b, : trees[b].n], acc.sequence(b))
        say(f"llama3-8b-chain2-b16 seq {b}: max rel err {st['max_rel']:.2e}, gated {st['gated']}/{st['total']}, "
            f"accept checked {st['accept_checked']}, L={st['L']}")
    v.close()


def test_full_size_draft_matches_oracle():
    """The draft of the Llama-3-8B shape (TGF with expansion 11008, one
    decoder layer, two heads: 0.42B parameters, the target's LM head), prefix
    2048: the passes of a 60-token depth-6 expansion (k = 10) checked against
    the oracle's draft pass on the same pass trees and input features."""
    import paper_2502_11018_amd as P
    from oracle import draft as od
    from workloads.configs import DRAFTS
    ds = DRAFTS["llama3-8b"]
    m = ds.target
    t0 = time.time()
    say("llama3-8b draft: weights on the GPU")
    mw_gpu = gen.make_weights(m, 0, device="cuda")
    dw_gpu = gen.make_draft_weights(ds, 3, device="cuda")
    P_len = 2048
    dm = P.DraftModel(ds, dw_gpu, mw_gpu, max_batch=1, max_tree=64, max_depth=63, kv_capacity=P_len + 64)
    k, v = gen.synthetic_kv(ds.layer, 0, 0, P_len, 5, "cuda")
    dm.write_prefix(0, k, v)
    kv = (k.double().cpu().numpy(), v.double().cpu().numpy())
    feat = gen.draft_root_features(m.d_model, 1, 11, "cuda")
    say(f"llama3-8b draft: GPU tree ({time.time() - t0:.0f}s)")
    n, tok, par, sc = dm.tree([P_len], [7], feat, ds.k, ds.depth, ds.n_total)
    assert n[0] == ds.n_total + 1
    # replay the GPU's own pass trees on both sides: a pass tree is the root
    # plus the nodes expanded so far; rebuild them from a fresh GPU expansion
    # run pass by pass (the same code path as griffin_draft_tree)
    say(f"llama3-8b draft: host copy for the oracle ({time.time() - t0:.0f}s)")
    ow = oracle.OracleWeights(mw_gpu.to("cpu"), cache=True)
    dow = od.DraftOracleWeights(dw_gpu.to("cpu"), ow)
    fr = None
    trees = [gen.Tree(np.array([7], np.int32), np.array([-1], np.int32))]
    worst, compared, total = 0.0, 0, 0
    for it in range(3):
        t = trees[-1]
        gtok, glp = dm.step([P_len], [t], feat, ds.k)
        feats = np.zeros((t.n, m.d_model))
        feats[0] = feat[0].double().cpu().numpy()
        for i in range(1, t.n):
            feats[i] = fr[t.parents[i]]
        say(f"llama3-8b draft: oracle pass {it} over {t.n} nodes ({time.time() - t0:.0f}s)")
        r = od.draft_forward(dow, t, feats, kv, P_len)
        fr = r.regress
        otok, _ = od.topk_logprobs(r.logits, ds.k)
        srt = np.sort(r.logits, axis=1)[:, ::-1]
        for i in range(t.n):
            total += 1
            full = r.logits[i] - (srt[i, 0] + np.log(np.exp(r.logits[i] - srt[i, 0]).sum()))
            worst = max(worst, float(np.max(np.abs(glp[0, i] - full[gtok[0, i]]))))
            if (-np.diff(srt[i, : ds.k + 1])).min() > 2e-3:
                compared += 1
                assert list(gtok[0, i]) == list(otok[i]), (it, i)
        # next pass tree: the expansion's frontier from the GPU's own proposals
        rows = [i for i in range(t.n) if t.depths()[i] == it]
        cand = [(float(glp[0, r_, j]), r_, int(gtok[0, r_, j])) for r_ in rows for j in range(ds.k)]
        best = sorted(range(len(cand)), key=lambda c: (-cand[c][0], c))[: ds.k]
        toks = list(t.tokens) + [cand[c][2] for c in best]
        pars = list(t.parents) + [cand[c][1] for c in best]
        trees.append(gen.Tree(np.array(toks, np.int32), np.array(pars, np.int32)))
    say(f"llama3-8b draft: log-prob error {worst:.2e}, tokens compared on {compared}/{total} rows "
        f"({time.time() - t0:.0f}s)")
    assert worst < 2e-3 and compared >= total // 2
    dm.close()


def test_full_size_cycle_is_lossless():
    """Whole draft-and-verify cycles at the Llama-3-8B shape (prefix 2048,
    the 0.42B draft with random weights, k 10, depth 6, 60 tokens): the
    emitted tokens equal the oracle's greedy continuation as far as its
    margins exceed the acceptance gate's 1e-2."""
    import paper_2502_11018_amd as P
    from paper_2502_11018_amd.cycle import SpeculativeCycle
    from workloads.configs import DRAFTS
    w = get_workload("llama3-8b")
    m, ds = w.model, DRAFTS["llama3-8b"]
    n_tokens, P_len = 8, w.prefix_len
    t0 = time.time()
    say("llama3-8b cycle: weights on the GPU")
    mw_gpu = gen.make_weights(m, w.weight_seed, device="cuda")
    cap = P_len + 64 + 64
    v = P.TreeVerifier(m, mw_gpu, max_batch=1, max_tree=64, max_depth=ds.depth, kv_capacity=cap)
    Ks, Vs = [], []
    for l in range(m.n_layers):
        k, vv = gen.synthetic_kv(m, l, 0, P_len, w.weight_seed, "cuda")
        v.write_prefix(l, 0, k, vv)
        Ks.append(k.to(torch.float64).cpu().numpy())
        Vs.append(vv.to(torch.float64).cpu().numpy())
    kv = H.PrefixKV(Ks, Vs)
    dm = P.DraftModel(ds, gen.make_draft_weights(ds, 3, device="cuda"), mw_gpu, max_batch=1, max_tree=64,
                      max_depth=ds.depth, kv_capacity=cap)
    dk, dv = gen.synthetic_kv(ds.layer, 0, 0, P_len, 5, "cuda")
    dm.write_prefix(0, dk, dv)
    root = 1234
    cyc = SpeculativeCycle(v, dm, ds.k, ds.depth, ds.n_total)
    cyc.start([P_len], [root], gen.draft_root_features(m.d_model, 1, 11, "cuda"))
    out = []
    while len(out) < n_tokens:
        say(f"llama3-8b cycle at prefix {cyc.prefix[0]} ({time.time() - t0:.0f}s)")
        out += cyc.cycle()[0]
    dm.close()
    v.close()
    say(f"llama3-8b cycle: oracle greedy continuation ({time.time() - t0:.0f}s)")
    ow = oracle.OracleWeights(mw_gpu.to("cpu"), cache=True)
    cache, tok, greedy, margins = kv.decode_cache(m), root, [], []
    for j in range(n_tokens):                       # oracle.greedy_chain, one token at a time (progress)
        logits = oracle.decode_step(ow, cache, tok, P_len + j)
        tok = int(oracle.argmax_first(logits))
        greedy.append(tok)
        margins.append(float(oracle.top2_margin(logits)))
        say(f"llama3-8b cycle: oracle token {j}: {tok} (margin {margins[-1]:.3f}, {time.time() - t0:.0f}s)")
    decided = next((i for i, mg in enumerate(margins) if mg <= H.MARGIN_GATE), n_tokens)
    say(f"llama3-8b cycle: {decided} tokens decided beyond the margin gate ({time.time() - t0:.0f}s)")
    assert decided >= 3
    assert out[:decided] == [int(t) for t in greedy[:decided]]
