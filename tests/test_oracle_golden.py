"""The oracle's acceptance walk and latency model against the hand-derived and
paper-printed fixtures in tests/golden/ (CPU only)."""

import os

import numpy as np
import pytest

import oracle
from workloads.gen import Tree

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def load_accept_cases():
    cases = []
    with open(os.path.join(GOLDEN, "accept_cases.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            name, par, tok, pred, L, acc, path = [c.strip() for c in line.split("|")]
            ints = lambda s: [int(v) for v in s.split()]  # noqa: E731
            cases.append(dict(name=name, parents=ints(par), tokens=ints(tok), pred=ints(pred),
                              L=int(L), accepted=ints(acc), path=ints(path)))
    return cases


ACCEPT_CASES = load_accept_cases()


@pytest.mark.parametrize("case", ACCEPT_CASES, ids=[c["name"] for c in ACCEPT_CASES])
def test_accept_walk_golden(case):
    tree = Tree(np.array(case["tokens"], dtype=np.int32), np.array(case["parents"], dtype=np.int32))
    res = oracle.accept_dfs(tree, case["pred"])
    assert res.length == case["L"]
    assert res.tokens == case["accepted"]
    assert res.path == case["path"]
    assert len(res.tokens) == res.length + 1


def test_latency_model_worked_example():
    with open(os.path.join(GOLDEN, "latency_example.txt")) as f:
        rows = [l for l in f if l.strip() and not l.startswith("#")]
    t, tb, d, tau, printed, prec = [float(x) for x in rows[0].split("|")]
    sr = oracle.speedup_ratio(t, tb, int(d), tau)
    assert abs(sr - printed) <= prec
    # and it is the ratio of the two total latencies
    n = 1000
    ratio = oracle.latency.total_latency(n, t) / oracle.latency.total_latency(n, t, tb, int(d), tau)
    assert abs(ratio - sr) < 1e-12
