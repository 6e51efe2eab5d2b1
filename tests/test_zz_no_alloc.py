"""The allocation-free stochastic walk (griffin_accept_sampled_walk_noalloc)
against the allocating one (griffin_accept_sampled_walk) through the C ABI:
the same kernels on the same inputs, so every output must be identical, on
two calls in a row (the second smaller, reusing the fixed block the first
left behind), and a call beyond the fixed block must fail before any device
work."""

import numpy as np
import pytest
import torch

from workloads import gen

pytestmark = pytest.mark.gpu


def say(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _pack(cases, max_tree, V):
    B = len(cases)
    lg = np.zeros((B * max_tree, V), np.float32)
    q = np.zeros((B * max_tree, V), np.float32)
    ua = np.zeros((B, max_tree), np.float32)
    uf = np.zeros((B, max_tree), np.float32)
    for b, c in enumerate(cases):
        n = c.tree.n
        lg[b * max_tree: b * max_tree + n] = c.logits
        q[b * max_tree: b * max_tree + n] = c.q
        ua[b, :n] = c.u_accept
        uf[b, :n] = c.u_final
    return torch.from_numpy(lg).cuda(), torch.from_numpy(q).cuda(), ua, uf


def _both(cases, V, T, max_tree, D):
    import paper_2502_11018_amd as P
    lg, q, ua, uf = _pack(cases, max_tree, V)
    trees = [c.tree for c in cases]
    ref = P.accept_sampled_walk(trees, lg, q, ua, uf, T, max_tree, D, V)
    got = P.accept_sampled_walk(trees, lg, q, ua, uf, T, max_tree, D, V, noalloc=True)
    assert np.array_equal(got.length, ref.length)
    assert np.array_equal(got.tokens, ref.tokens)
    assert np.array_equal(got.path, ref.path)
    return ref


def test_noalloc_walk_equals_the_allocating_walk():
    # first call: Llama-3 vocabulary, 60-node trees, batch 6
    say("noalloc walk: V=128256 batch 6")
    big = [gen.sampled_case((10,) * 6, 128256, 700 + 13 * i, temperature=1.0) for i in range(6)]
    r1 = _both(big, 128256, 1.0, 64, 6)
    # second call, smaller: it reuses the block the first one left behind
    say("noalloc walk: V=3000 batch 2, after the larger call")
    small = [gen.sampled_case((3, 3, 2), 3000, 900 + 7 * i, temperature=0.7) for i in range(2)]
    r2 = _both(small, 3000, 0.7, 16, 3)
    say(f"noalloc walk: lengths {list(r1.length)} then {list(r2.length)}")
    assert r1.length.sum() > 0


def test_noalloc_walk_rejects_work_beyond_its_block():
    import paper_2502_11018_amd as P
    B, max_tree, V = 40, 64, 131072       # about 6.7 MB of device memory: above the 4 MiB block
    say("noalloc walk: beyond the fixed block")
    lg = torch.zeros((B * max_tree, V), dtype=torch.float32, device="cuda")
    trees = [gen.chain_tree(1, [2]) for _ in range(B)]
    u = np.full((B, max_tree), 0.5, np.float32)
    with pytest.raises(P.GriffinError) as ei:
        P.accept_sampled_walk(trees, lg, lg, u, u, 1.0, max_tree, 1, V, noalloc=True)
    assert ei.value.name == "GRIFFIN_ENOMEM"
    del lg
    torch.cuda.synchronize()
