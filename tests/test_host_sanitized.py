"""The host planning code (tree validation and metadata, the prefix-attention
split table, model-shape checks, the stochastic acceptance's work list) built
into a CPU program with the address and undefined-behaviour sanitizers
(tests/host_plan_check.cpp), driven with edge cases and random cases whose
results are checked here against plain Python."""

import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle.verify import ancestor_matrix
from workloads.configs import WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OK, EINVAL, ESHAPE, ETREE, ETOKEN, ECAPACITY = 0, -1, -2, -3, -4, -5


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp("hpc") / "host_plan_check")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-fno-omit-frame-pointer", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2502_11018_amd", "csrc"),
           os.path.join(ROOT, "tests", "host_plan_check.cpp"),
           os.path.join(ROOT, "paper_2502_11018_amd", "csrc", "plan.cpp"), "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)

    def run(lines):
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
                   UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
        p = subprocess.run([exe], input="\n".join(lines) + "\n", capture_output=True, text=True, env=env,
                           timeout=120)
        assert p.returncode == 0 and "runtime error" not in p.stderr and "Sanitizer" not in p.stderr, p.stderr
        out = p.stdout.splitlines()
        assert len(out) == len(lines)
        return out
    return run


def _tree_line(tok, par, prefix=10, mt=64, md=63, vocab=1000, cap=4096):
    n = len(tok)
    return " ".join(map(str, ["T", n, prefix, mt, md, vocab, cap, *tok, *par]))


def _random_tree(rng, n):
    par = [-1] + [int(rng.integers(0, i)) for i in range(1, n)]
    return [int(t) for t in rng.integers(0, 1000, n)], par


def test_tree_preparation_matches_python(driver):
    rng = np.random.default_rng(3)
    cases, lines = [], []
    for n in [1, 2, 7, 33, 63, 64]:
        for _ in range(3):
            tok, par = _random_tree(rng, n)
            cases.append((tok, par))
            lines.append(_tree_line(tok, par, prefix=int(rng.integers(0, 3000))))
    star = ([5] * 64, [-1] + [0] * 63)
    chain = (list(range(64)), [-1] + list(range(63)))
    cases += [star, chain]
    lines += [_tree_line(*star), _tree_line(*chain)]
    out = driver(lines)
    for (tok, par), line, res in zip(cases, lines, out):
        v = [int(x) for x in res.split()]
        n = len(tok)
        prefix = int(line.split()[2])
        assert v[0] == OK
        depth, pos, anc = v[1: 1 + n], v[1 + n: 1 + 2 * n], v[1 + 2 * n:]
        vis = ancestor_matrix(np.array(par))
        want_depth = vis.sum(axis=1) - 1
        assert depth == list(want_depth) and pos == [prefix + d for d in want_depth]
        for i in range(n):
            assert anc[i] == sum(1 << j for j in range(n) if vis[i, j])


def test_tree_preparation_rejects(driver):
    tok, par = list(range(6)), [-1, 0, 0, 1, 2, 3]
    bad = [
        (_tree_line(tok, [0] + par[1:]), ETREE),                    # root with a parent
        (_tree_line(tok, par[:3] + [3] + par[4:]), ETREE),          # parent not before the node
        (_tree_line(tok, par[:3] + [-5] + par[4:]), ETREE),         # negative parent
        (_tree_line(tok[:2] + [1000] + tok[3:], par), ETOKEN),      # token = vocab
        (_tree_line(tok[:2] + [-1] + tok[3:], par), ETOKEN),
        (_tree_line(tok, par, md=2), ETREE),                        # depth 3 > max_depth
        (_tree_line(tok, par, mt=5), ETREE),                        # n > max_tree
        (_tree_line(tok, par, prefix=4091, cap=4096), ECAPACITY),   # prefix + n > capacity
        (_tree_line(tok, par, prefix=-1), ECAPACITY),
        (_tree_line(list(range(65)), [-1] + list(range(64)), mt=80, md=79), ETREE),   # above 64 nodes
        ("T 0 10 64 63 1000 4096", ETREE),                          # empty tree
    ]
    out = driver([l for l, _ in bad])
    for (line, code), res in zip(bad, out):
        assert int(res.split()[0]) == code, line
    # the boundary cases that are valid
    ok = driver([_tree_line(tok, par, prefix=4090, cap=4096), _tree_line(tok, par, md=3), _tree_line(tok, par, mt=6)])
    assert all(int(r.split()[0]) == OK for r in ok)


def test_split_plan_invariants(driver):
    rng = np.random.default_rng(11)
    cases = []
    for _ in range(200):
        batch = int(rng.integers(1, 17))
        splits = int(rng.integers(1, 17))
        sp = int(rng.integers(splits, 2 * splits + 1))
        prefix = [int(x) for x in rng.integers(0, 20000, batch)]
        if rng.random() < 0.2:
            prefix[0] = 0
        nodes = [int(x) for x in rng.integers(1, 65, batch)]
        cases.append((batch, splits, sp, prefix, nodes))
    out = driver([" ".join(map(str, ["S", b, s, sp, *p, *n])) for b, s, sp, p, n in cases])
    for (batch, splits, sp, prefix, nodes), res in zip(cases, out):
        v = [int(x) for x in res.split()]
        tab = np.array(v[: 4 * batch * splits]).reshape(-1, 4)
        nsplit, slots = v[4 * batch * splits:-1], v[-1]
        assert len(nsplit) == batch and sum(nsplit) <= batch * splits
        # the merge reads the first `slots` partial slots: every split, within the allocation
        assert max(nsplit) <= slots <= sp
        assert slots == sp or (slots & (slots - 1)) == 0 and slots < 2 * max(nsplit)
        j = 0
        for b in range(batch):
            cap = max(1, min(sp, ((prefix[b] + 31) // 32) // 2))
            assert 1 <= nsplit[b] <= cap
            for s in range(nsplit[b]):
                assert list(tab[j]) == [b | (s << 16), nsplit[b], prefix[b], nodes[b]]
                j += 1
        assert all(list(t) == [-1, 0, 0, 0] for t in tab[j:])


def test_model_shape_validation(driver):
    def line(m, **kw):
        f = dict(n_layers=m.n_layers, d_model=m.d_model, hq=m.n_q_heads, hkv=m.n_kv_heads, dh=m.head_dim,
                 d_ff=m.d_ff, vocab=m.vocab, experts=m.n_experts, top_k=m.top_k, eps=m.rms_eps,
                 base=m.rope_base, mb=1, mt=64, md=6, cap=4096)
        f.update(kw)
        return "D " + " ".join(str(f[k]) for k in ["n_layers", "d_model", "hq", "hkv", "dh", "d_ff", "vocab",
                                                   "experts", "top_k", "eps", "base", "mb", "mt", "md", "cap"])
    models = sorted({w.model for w in WORKLOADS.values()}, key=lambda m: m.name)
    good = [line(m) for m in models]
    assert all(int(r) == OK for r in driver(good))
    m = models[0]
    bad = [line(m, dh=96), line(m, hq=6, hkv=4), line(m, d_model=8200), line(m, experts=65),
           line(m, experts=8, top_k=5), line(m, experts=8, top_k=0), line(m, mt=65), line(m, mt=0),
           line(m, md=64), line(m, md=-1), line(m, cap=100), line(m, cap=0), line(m, eps=0), line(m, base=1),
           line(m, mb=0), line(m, d_ff=100), line(m, n_layers=0)]
    assert all(int(r) == ESHAPE for r in driver(bad))


def test_sampled_work_list_matches_python(driver):
    rng = np.random.default_rng(5)
    lines, cases = [], []
    for _ in range(40):
        batch, mt = int(rng.integers(1, 6)), 64
        nodes = [int(x) for x in rng.integers(1, mt + 1, batch)]
        par = np.zeros((batch, mt), np.int32)
        tok = rng.integers(0, 1000, (batch, mt)).astype(np.int32)
        for b in range(batch):
            par[b, 0] = -1
            for i in range(1, nodes[b]):
                par[b, i] = rng.integers(0, i)
        cases.append((batch, mt, nodes, par, tok))
        lines.append(" ".join(map(str, ["Q", batch, mt, *nodes, *par.ravel(), *tok.ravel()])))
    for (batch, mt, nodes, par, tok), res in zip(cases, driver(lines)):
        parts = [[int(x) for x in p.split()] for p in res.split("|")]
        kids = {b * mt + i: [] for b in range(batch) for i in range(nodes[b])}
        for b in range(batch):
            for i in range(1, nodes[b]):
                kids[b * mt + par[b, i]].append(i)
        order = sorted(kids, key=lambda r: (-len(kids[r]), r))       # stable by row
        cmax = len(kids[order[0]])
        rows_with = [sum(len(kids[r]) >= j for r in order) for j in range(cmax + 1)]
        child, token = [], []
        for k in range(cmax):
            for r in order[: rows_with[k + 1]]:
                child.append(kids[r][k])
                token.append(int(tok[r // mt, kids[r][k]]))
        assert parts == [order, rows_with, child, token]
