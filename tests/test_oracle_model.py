"""Pins of the oracle's tree-verification pass and acceptance walk against
plain causal decoding, brute force, closed forms and invariants (CPU only)."""

from dataclasses import replace

import numpy as np
import pytest
import torch

import oracle
from oracle import model as om
from oracle.verify import ancestor_matrix
from workloads import gen
from workloads.configs import Workload, get_workload
from tests.harness import build_sequence, micro_shape, prefix_kv_prefill, PrefixKV


def _model(shape, seed=0):
    mw = gen.make_weights(shape, seed)
    return mw, oracle.OracleWeights(mw)


@pytest.fixture(scope="module")
def micro():
    shape = micro_shape()
    mw, ow = _model(shape)
    toks = gen.prefix_tokens(Workload("m", shape, 1, 11, (2, 2), "leaf", "prefill"))
    kv = prefix_kv_prefill(ow, toks)
    return shape, mw, ow, kv


def _verify(ow, kv: PrefixKV, tree):
    return oracle.verify_tree(ow, kv.fn(), tree, kv.length)


# ----------------------------------------------------- decoding equivalences ----

def test_chain_tree_equals_causal_decoding(micro):
    shape, _, ow, kv = micro
    toks = [5, 17, 3, 88, 41, 9]
    tree = gen.chain_tree(60, toks)
    res = _verify(ow, kv, tree)
    cache = kv.decode_cache(shape)
    for i, t in enumerate([60] + toks):
        ref = oracle.decode_step(ow, cache, t, kv.length + i)
        np.testing.assert_allclose(res.logits[i], ref, rtol=1e-10, atol=1e-10)


def test_single_node_tree_equals_decode_step(micro):
    shape, _, ow, kv = micro
    tree = gen.chain_tree(33, [])
    res = _verify(ow, kv, tree)
    ref = oracle.decode_step(ow, kv.decode_cache(shape), 33, kv.length)
    np.testing.assert_allclose(res.logits[0], ref, rtol=1e-11, atol=1e-11)


def test_every_node_equals_decoding_its_root_path(micro):
    shape, _, ow, kv = micro
    tree, _ = gen.random_tree((3, 3, 4, 2), shape.vocab, seed=77)
    res = _verify(ow, kv, tree)
    for i in range(tree.n):
        cache = kv.decode_cache(shape)
        nodes = [0] + tree.root_path(i)
        for depth, n in enumerate(nodes):
            ref = oracle.decode_step(ow, cache, int(tree.tokens[n]), kv.length + depth)
        np.testing.assert_allclose(res.logits[i], ref, rtol=1e-10, atol=1e-10)


def test_tree_keys_are_node_keys_at_depth_positions(micro):
    # the K/V a node contributes equal what decoding its root path appends
    shape, _, ow, kv = micro
    tree, _ = gen.random_tree((2, 3), shape.vocab, seed=5)
    res = _verify(ow, kv, tree)
    i = tree.n - 1
    cache = kv.decode_cache(shape)
    for depth, n in enumerate([0] + tree.root_path(i)):
        oracle.decode_step(ow, cache, int(tree.tokens[n]), kv.length + depth)
    for l in range(shape.n_layers):
        np.testing.assert_allclose(res.tree_k[l][i], cache.K[l][:, -1, :], rtol=1e-11, atol=1e-11)
        np.testing.assert_allclose(res.tree_v[l][i], cache.V[l][:, -1, :], rtol=1e-11, atol=1e-11)


# ------------------------------------------------------------- invariants ----

def test_mask_isolation_is_bit_exact(micro):
    shape, _, ow, kv = micro
    tree, _ = gen.random_tree((3, 3, 3), shape.vocab, seed=9)
    base = _verify(ow, kv, tree).logits
    vis = ancestor_matrix(tree.parents)
    for i in [1, 4, tree.n - 1]:
        t2 = tree.copy()
        others = [j for j in range(1, tree.n) if not vis[i, j]]
        for j in others:
            t2.tokens[j] = (t2.tokens[j] + 1 + j) % shape.vocab
        out = _verify(ow, kv, t2).logits
        np.testing.assert_array_equal(out[i], base[i])
        changed = [j for j in others if not np.array_equal(out[j], base[j])]
        assert changed, "changing a node's token must change its own logits"


def test_node_relabelling_permutes_logits(micro):
    shape, _, ow, kv = micro
    tree, _ = gen.random_tree((3, 4, 3), shape.vocab, seed=21)
    res = _verify(ow, kv, tree)
    # depth-first numbering of the same tree keeps parent < child
    children = {i: [] for i in range(tree.n)}
    for i in range(1, tree.n):
        children[int(tree.parents[i])].append(i)
    order, stack = [], [0]
    while stack:
        n = stack.pop()
        order.append(n)
        stack.extend(reversed(children[n]))
    new_id = {old: new for new, old in enumerate(order)}
    t2 = gen.Tree(tree.tokens[order].copy(),
                  np.array([-1] + [new_id[int(tree.parents[o])] for o in order[1:]], dtype=np.int32))
    assert all(t2.parents[i] < i for i in range(1, t2.n))
    res2 = _verify(ow, kv, t2)
    np.testing.assert_allclose(res2.logits, res.logits[order], rtol=1e-11, atol=1e-11)


def test_gqa_equals_mha_with_duplicated_kv_heads(micro):
    shape, mw, ow, kv = micro
    G = shape.n_q_heads // shape.n_kv_heads
    mha = replace(shape, n_kv_heads=shape.n_q_heads)
    dh, Hq = shape.head_dim, shape.n_q_heads
    layers = []
    for L in mw.layers:
        w = L["w_qkv"]
        q = w[: Hq * dh]
        k = w[Hq * dh: (Hq + shape.n_kv_heads) * dh].view(shape.n_kv_heads, dh, -1)
        v = w[(Hq + shape.n_kv_heads) * dh:].view(shape.n_kv_heads, dh, -1)
        k2 = k.repeat_interleave(G, dim=0).reshape(Hq * dh, -1)
        v2 = v.repeat_interleave(G, dim=0).reshape(Hq * dh, -1)
        L2 = dict(L)
        L2["w_qkv"] = torch.cat([q, k2, v2], dim=0)
        layers.append(L2)
    mw2 = gen.ModelWeights(mha, mw.embed, mw.lm_head, mw.final_norm, layers)
    ow2 = oracle.OracleWeights(mw2)
    kv2 = PrefixKV([np.repeat(k, G, axis=0) for k in kv.K], [np.repeat(v, G, axis=0) for v in kv.V])
    tree, _ = gen.random_tree((2, 3, 2), shape.vocab, seed=3)
    np.testing.assert_allclose(_verify(ow2, kv2, tree).logits, _verify(ow, kv, tree).logits,
                               rtol=1e-11, atol=1e-11)


def test_moe_with_identical_experts_equals_dense_model(micro):
    shape, mw, ow, kv = micro
    E = 4
    moe_shape = replace(shape, n_experts=E, top_k=2)
    layers = []
    for l, L in enumerate(mw.layers):
        L2 = dict(L)
        L2["w_gate_up"] = L["w_gate_up"].unsqueeze(0).repeat(E, 1, 1)
        L2["w_down"] = L["w_down"].unsqueeze(0).repeat(E, 1, 1)
        L2["w_router"] = gen.hashed_normal_bf16(E * shape.d_model, 5, 900 + l, 0.02).view(E, -1)
        layers.append(L2)
    ow2 = oracle.OracleWeights(gen.ModelWeights(moe_shape, mw.embed, mw.lm_head, mw.final_norm, layers))
    tree, _ = gen.random_tree((2, 2), shape.vocab, seed=4)
    np.testing.assert_allclose(_verify(ow2, kv, tree).logits, _verify(ow, kv, tree).logits,
                               rtol=1e-11, atol=1e-11)


# ---------------------------------------------------------- closed forms ----

def test_zero_layers_pass_embedding_through_residual():
    shape = micro_shape()
    mw, _ = _model(shape)
    layers = [{k: (None if v is None else torch.zeros_like(v)) for k, v in L.items()} for L in mw.layers]
    for L in layers:
        L["attn_norm"] = torch.ones_like(L["attn_norm"])
        L["mlp_norm"] = torch.ones_like(L["mlp_norm"])
    ow = oracle.OracleWeights(gen.ModelWeights(shape, mw.embed, mw.lm_head, mw.final_norm, layers))
    kv = PrefixKV([np.zeros((shape.n_kv_heads, 4, shape.head_dim))] * shape.n_layers,
                  [np.zeros((shape.n_kv_heads, 4, shape.head_dim))] * shape.n_layers)
    tree = gen.chain_tree(7, [8, 9])
    out = _verify(ow, kv, tree).logits
    E = mw.embed.to(torch.float64).numpy()
    W = mw.lm_head.to(torch.float64).numpy()
    g = mw.final_norm.to(torch.float64).numpy()
    assert np.ptp(g) > 0          # a non-unit final gain, applied per column
    x = E[[7, 8, 9]]
    want = (x / np.sqrt(np.mean(x * x, axis=1, keepdims=True) + shape.rms_eps) * g) @ W.T
    np.testing.assert_allclose(out, want, rtol=1e-12, atol=1e-12)


def test_one_token_no_prefix_reduces_to_attention_free_formula():
    # a lone token attends only to itself, so its attention output is its own
    # value vector per head: no softmax, no rotation enters the result
    shape = micro_shape(n_layers=1)
    mw, ow = _model(shape, seed=3)
    empty = np.zeros((shape.n_kv_heads, 0, shape.head_dim))
    kv = PrefixKV([empty], [empty])
    out = _verify(ow, kv, gen.chain_tree(11, [])).logits[0]
    L = ow.layer(0)
    m = shape
    x = ow.embed([11])
    h = om.rmsnorm(x, L["attn_norm"], m.rms_eps)
    _, _, v = om.split_qkv(h, L["w_qkv"], m)
    o = np.repeat(v[0], m.n_q_heads // m.n_kv_heads, axis=0).reshape(1, -1)
    x = x + o @ L["w_o"].T
    x = x + om.swiglu(om.rmsnorm(x, L["mlp_norm"], m.rms_eps), L["w_gate_up"], L["w_down"])
    want = (om.rmsnorm(x, ow.final_norm, m.rms_eps) @ ow.lm_head().T)[0]
    np.testing.assert_allclose(out, want, rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------- acceptance ----

@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_accept_dfs_equals_brute_force_and_trie(micro, seed):
    shape, _, ow, kv = micro
    tree, _ = gen.random_tree((3, 3, 3, 2), shape.vocab, seed=100 + seed)
    greedy, margins, _ = oracle.greedy_chain(ow, kv.decode_cache(shape), int(tree.tokens[0]), 5)
    # plant greedy prefixes of different lengths on a few branches so that
    # the walk has work to do
    r = np.random.default_rng(seed)
    for node in r.choice(np.arange(1, tree.n), size=4, replace=False):
        path = tree.root_path(int(node))
        keep = int(r.integers(0, len(path) + 1))
        tree = gen.apply_plant(tree, path[:keep], greedy)
    res = _verify(ow, kv, tree)
    pred = oracle.argmax_first(res.logits)
    dfs = oracle.accept_dfs(tree, pred)
    bf = oracle.brute_force_accept(ow, kv.decode_cache(shape), tree)
    assert (dfs.length, dfs.tokens) == (bf.length, bf.tokens)
    assert dfs.length == oracle.accept_trie(tree, greedy)
    # the emitted tokens are the target's own greedy continuation (losslessness)
    assert dfs.tokens == greedy[: dfs.length + 1]
    depth = tree.depths()
    assert 0 <= dfs.length <= depth.max()


def test_tiny_workload_planted_paths_fully_accepted():
    w = get_workload("tiny")
    mw, ow = _model(w.model, w.weight_seed)
    kv = prefix_kv_prefill(ow, gen.prefix_tokens(w))
    for ti in range(3):
        case = build_sequence(ow, w, ti, kv=kv)
        res = _verify(ow, kv, case.tree)
        acc = oracle.accept_dfs(case.tree, oracle.argmax_first(res.logits))
        assert acc.length >= len(case.plant_path)
        assert acc.tokens[: len(case.greedy)] == case.greedy
        assert acc.length <= w.depth


def test_top2_margin():
    x = np.array([[1.0, 5.0, 4.5, -2.0], [3.0, 3.0, 1.0, 0.0]])
    np.testing.assert_allclose(oracle.top2_margin(x), [0.5, 0.0])
    assert list(oracle.argmax_first(x)) == [1, 0]
