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
    import paper_2502_11018_amd as P
    w = get_workload(name)
    m = w.model
    t0 = time.time()
    say(f"{name}: generate weights on the GPU")
    mw_gpu = gen.make_weights(m, w.weight_seed, device="cuda")
    v = P.TreeVerifier(m, mw_gpu, max_batch=1, max_tree=64, max_depth=w.depth, kv_capacity=w.kv_capacity())
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
        st = H.check_parity(os_, lg, pred[: tree.n], acc.sequence(0))
        rel = np.abs(lg - os_.logits).max(axis=1)
        say(f"{name} {label}: max rel err {st['max_rel']:.2e}, max abs err {rel.max():.3e}, "
            f"gated {st['gated']}/{st['total']}, accept checked {st['accept_checked']}, L={st['L']}")
        if label.startswith("planted") and st["accept_checked"]:
            assert int(acc.length[0]) >= len(path)
    v.close()
