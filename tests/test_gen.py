"""Seeded input generators (CPU only)."""

import numpy as np
import pytest
import torch

from workloads import gen
from workloads.configs import WORKLOADS, get_workload


def test_mix32_matches_python_integer_definition():
    xs = [0, 1, 2, 0x7FFFFFFF, 0x80000000, 0xFFFFFFFF, 123456789, 0xDEADBEEF]
    t = gen.mix32(torch.tensor(xs, dtype=torch.int64))
    assert [int(v) for v in t] == [gen._mix32_int(x) for x in xs]
    # lowbias32 is a bijection with 0 as a fixed point
    assert gen._mix32_int(0) == 0


def test_hashed_normal_is_deterministic_chunk_independent_and_scaled():
    a = gen.hashed_normal_bf16(300000, seed=3, stream=7, std=0.02)
    b = gen.hashed_normal_bf16(300000, seed=3, stream=7, std=0.02)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    part = gen.hashed_normal_bf16(1000, seed=3, stream=7, std=0.02, start=123456)
    assert torch.equal(part.view(torch.int16), a[123456:124456].view(torch.int16))
    other = gen.hashed_normal_bf16(1000, seed=3, stream=8, std=0.02)
    assert not torch.equal(other, a[:1000])
    x = a.to(torch.float64)
    assert abs(x.mean().item()) < 2e-4
    assert abs(x.std().item() - 0.02) < 2e-4
    assert x.abs().max().item() <= 0.02 * 3.47


def test_make_weights_shapes_and_layouts():
    w = get_workload("small-moe").model
    mw = gen.make_weights(w, 0)
    L = mw.layers[0]
    assert L["w_qkv"].shape == (w.qkv_rows, w.d_model)
    assert L["w_gate_up"].shape == (w.n_experts, 2 * w.d_ff, w.d_model)
    assert L["w_down"].shape == (w.n_experts, w.d_model, w.d_ff)
    assert L["w_router"].shape == (w.n_experts, w.d_model)
    assert mw.embed.dtype == torch.bfloat16
    # RMSNorm gains: 1 + N(0, 0.1^2), bounded, and different per layer and norm
    gains = [L["attn_norm"], L["mlp_norm"], mw.layers[1]["attn_norm"], mw.final_norm]
    for g in gains:
        assert g.shape == (w.d_model,) and g.dtype == torch.bfloat16
        dev = g.float() - 1.0
        assert 0.08 < dev.std().item() < 0.12 and dev.abs().max().item() <= 0.1 * 3.47
    for i in range(len(gains)):
        for j in range(i):
            assert not torch.equal(gains[i], gains[j])
    # storage = what a pass streams + the embedding table (only T rows of it are read)
    assert mw.nbytes() == w.weight_bytes() + 2 * w.vocab * w.d_model


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_workload_trees(name):
    w = WORKLOADS[name]
    for b in sorted({0, 1, w.batch - 1} & set(range(w.batch))) if not w.seq_widths else range(w.batch):
        widths = w.widths_of(b)
        for i in range(4):
            tree, path = gen.workload_tree(w, i, b)
            assert tree.n == 1 + sum(widths) <= w.tree_nodes <= w.max_tree
            assert tree.parents[0] == -1
            d = tree.depths()
            for j in range(1, tree.n):
                assert 0 <= tree.parents[j] < j
            # breadth-first numbering with the configured widths
            assert [int((d == k).sum()) for k in range(1, len(widths) + 1)] == list(widths)
            assert np.all(np.diff(d) >= 0)
            assert tree.tokens.min() >= 0 and tree.tokens.max() < w.model.vocab
            # the planting path is a root path
            for k, node in enumerate(path):
                assert d[node] == k + 1
                if k:
                    assert tree.parents[node] == path[k - 1]
            if w.plant == "leaf" and tree.n > 1:
                assert path and not any(tree.parents[j] == path[-1] for j in range(1, tree.n))
            tree2, path2 = gen.workload_tree(w, i, b)
            assert np.array_equal(tree.tokens, tree2.tokens) and path == path2


def test_half_planting_rate_and_lengths():
    w = get_workload("llama3-8b")
    lengths = [len(gen.workload_tree(w, i)[1]) for i in range(400)]
    planted = [l for l in lengths if l > 0]
    # Bernoulli(1/2) to plant, then a length uniform on 0..6 (0 plants nothing)
    frac = sum(1 for i in range(400) if gen.workload_tree(w, i)[1] or False) / 400
    assert 0.33 < frac < 0.52
    assert max(planted) == 6 and min(planted) >= 1


def test_apply_plant_and_chain_tree():
    t = gen.chain_tree(4, [5, 6, 7])
    assert list(t.parents) == [-1, 0, 1, 2]
    assert list(t.depths()) == [0, 1, 2, 3]
    t2 = gen.apply_plant(t, [1, 2], [9, 8])
    assert list(t2.tokens) == [4, 9, 8, 7]
    assert list(t.tokens) == [4, 5, 6, 7]


def test_synthetic_kv_scale_and_determinism():
    m = get_workload("small-gqa").model
    k, v = gen.synthetic_kv(m, 1, 0, 50)
    k2, _ = gen.synthetic_kv(m, 1, 0, 50)
    assert k.shape == (m.n_kv_heads, 50, m.head_dim)
    assert torch.equal(k, k2)
    assert not torch.equal(k, v)
    assert abs(k.float().std().item() - gen.kv_std(m)) < 0.03 * gen.kv_std(m)


def test_ragged_batch_workloads():
    """Per-sequence prefixes and tree sizes: prefix tokens and the KV capacity
    follow each sequence's own length."""
    w = WORKLOADS["small-chain2"]
    P = w.prefixes()
    assert len(P) == w.batch == 16 and len(set(P)) > 8 and min(P) >= 20 and max(P) <= 200
    assert w.kv_capacity() >= max(P) + w.tree_nodes
    sizes = [1 + sum(w.widths_of(b)) for b in range(w.batch)]
    assert sorted(set(sizes)) == [1, 2, 3] and w.tree_nodes == 3 == w.max_tree
    for b in (0, 3, 15):
        assert len(gen.prefix_tokens(w, b)) == P[b]
    for B in (2, 4, 8, 16):
        c = WORKLOADS[f"llama3-8b-chain2-b{B}"]
        assert c.batch == B and c.max_tree == 3 and c.depth == 2
        assert all(256 <= p <= 2048 for p in c.prefixes())
