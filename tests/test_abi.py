"""The C ABI library on the CPU: it loads, exports every function the header
declares, and its host-only validation and tree metadata are right (no device
work is done here)."""

import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "griffin_verify.h")


def _native():
    from paper_2502_11018_amd import build as B
    if not os.path.exists(os.path.join(B.LIBDIR, B.LIBNAME)):
        B.build()
    from paper_2502_11018_amd import _native as N
    return N


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(griffin_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    N = _native()
    declared = header_functions()
    assert len(declared) >= 10
    lib = ctypes.CDLL(N.LIB_PATH)
    for name in declared:
        assert hasattr(lib, name), f"{name} declared in the header but not exported"
    assert sorted(N.EXPORTED) == declared


def test_kernel_classes_match_header():
    """The binding's class names line up with the header's GRIFFIN_KC_* indices."""
    N = _native()
    text = open(HEADER).read()
    idx = {m[0]: int(m[1]) for m in re.findall(r"#define GRIFFIN_KC_([A-Z_]+) (\d+)", text)}
    assert idx.pop("COUNT") == len(N.KERNEL_CLASSES)
    assert sorted(idx.values()) == list(range(len(N.KERNEL_CLASSES)))
    expect = {"QKV": "qkv_gemm", "ROPE": "rope_kv_write", "ATTN": "tree_attention", "O": "o_gemm",
              "NORM": "residual_rmsnorm", "GATE_UP": "gate_up_gemm", "DOWN": "down_gemm",
              "LM_HEAD": "lm_head_gemm", "OTHER": "argmax_accept_route", "MERGE": "attn_merge"}
    for k, i in idx.items():
        assert N.KERNEL_CLASSES[i] == expect[k]


def test_status_strings():
    N = _native()
    for code in N.STATUS:
        s = N.lib.griffin_status_str(code).decode()
        assert s and s != "unknown status"
    assert N.lib.griffin_status_str(12345).decode() == "unknown status"


def _prep(tokens, parents, prefix=10, max_tree=64, max_depth=8, vocab=100, cap=128):
    from paper_2502_11018_amd.verifier import tree_prepare
    _native()
    return tree_prepare(tokens, parents, prefix, max_tree, max_depth, vocab, cap)


def test_tree_prepare_metadata_matches_python():
    from oracle.verify import ancestor_matrix
    from workloads import gen
    for seed in range(5):
        tree, _ = gen.random_tree((3, 5, 8, 8, 6, 5), 1000, seed)
        rc, depth, pos, anc = _prep(tree.tokens, tree.parents, prefix=37, vocab=1000, cap=128)
        assert rc == 0
        np.testing.assert_array_equal(depth, tree.depths())
        np.testing.assert_array_equal(pos, 37 + tree.depths())
        vis = ancestor_matrix(tree.parents)
        for i in range(tree.n):
            bits = {j for j in range(tree.n) if (int(anc[i]) >> j) & 1}
            assert bits == set(np.nonzero(vis[i])[0])


def test_tree_prepare_accepts_full_64_node_star():
    tokens = np.arange(64) % 50
    parents = np.array([-1] + [0] * 63)
    rc, depth, _, anc = _prep(tokens, parents, max_depth=1, vocab=50, cap=128)
    assert rc == 0 and depth.max() == 1
    assert int(anc[63]) == (1 << 63) | 1


@pytest.mark.parametrize("tokens,parents,kw,code", [
    ([1, 2], [0, 0], {}, "GRIFFIN_ETREE"),            # root parent must be -1
    ([1, 2, 3], [-1, 0, 2], {}, "GRIFFIN_ETREE"),     # parent not before the node
    ([1, 2, 3], [-1, 0, 5], {}, "GRIFFIN_ETREE"),     # parent out of range
    ([1, 2, 3], [-1, -1, 0], {}, "GRIFFIN_ETREE"),    # second root
    ([1, 2, 3, 4], [-1, 0, 1, 2], {"max_depth": 2}, "GRIFFIN_ETREE"),   # too deep
    (list(range(65)), [-1] + [0] * 64, {"max_depth": 1}, "GRIFFIN_ETREE"),  # more than 64 nodes
    ([1, 2, 3], [-1, 0, 0], {"max_tree": 2}, "GRIFFIN_ETREE"),
    ([1, 100, 3], [-1, 0, 0], {}, "GRIFFIN_ETOKEN"),
    ([1, -3, 3], [-1, 0, 0], {}, "GRIFFIN_ETOKEN"),
    ([1, 2, 3], [-1, 0, 0], {"prefix": 126}, "GRIFFIN_ECAPACITY"),
    ([1, 2, 3], [-1, 0, 0], {"prefix": -1}, "GRIFFIN_ECAPACITY"),
])
def test_tree_prepare_rejects(tokens, parents, kw, code):
    N = _native()
    rc, *_ = _prep(tokens, parents, **kw)
    assert rc == N.CODES[code]


def test_init_and_step_reject_bad_arguments_before_any_device_work():
    N = _native()
    from ctypes import byref, c_void_p
    ctx = c_void_p()
    # null descriptor / weights / caches
    assert N.lib.griffin_verify_init(None, None, None, None, None, byref(ctx)) == N.CODES["GRIFFIN_EINVAL"]
    desc = N.ModelDesc(2, 256, 4, 4, 96, 688, 1024, 1, 1, 1e-6, 1e4, 1, 16, 4, 192)  # head_dim 96
    w = N.Weights()
    assert N.lib.griffin_verify_init(byref(desc), byref(w), c_void_p(16), c_void_p(32), None, byref(ctx)) \
        == N.CODES["GRIFFIN_ESHAPE"]
    desc.head_dim = 64
    desc.kv_capacity = 100   # not a multiple of 32
    assert N.lib.griffin_verify_init(byref(desc), byref(w), c_void_p(16), c_void_p(32), None, byref(ctx)) \
        == N.CODES["GRIFFIN_ESHAPE"]
    desc.kv_capacity = 192
    # valid shape, null weight pointers
    assert N.lib.griffin_verify_init(byref(desc), byref(w), c_void_p(16), c_void_p(32), None, byref(ctx)) \
        == N.CODES["GRIFFIN_EINVAL"]
    assert not ctx.value
    assert N.lib.griffin_verify_step(None, 1, None, None, None, None, None) == N.CODES["GRIFFIN_EINVAL"]
    assert N.lib.griffin_accept(None, None, None, None) == N.CODES["GRIFFIN_EINVAL"]
    assert N.lib.griffin_kv_cache_bytes(byref(desc)) == 2 * 1 * 4 * 192 * 64 * 2
    N.lib.griffin_verify_free(None)


def test_sampled_cycle_rejects_bad_temperatures():
    """SpeculativeCycle validates its temperature before touching the GPU."""
    from paper_2502_11018_amd.cycle import SpeculativeCycle

    class _Stub:
        max_tree, max_batch = 64, 1

    for bad in (-1.0, float("nan"), float("inf")):
        with pytest.raises(ValueError):
            SpeculativeCycle(_Stub(), _Stub(), 10, 6, 60, temperature=bad)
    with pytest.raises(ValueError):     # the verifier cannot hold n_total + 1 nodes
        small = _Stub()
        small.max_tree = 16
        SpeculativeCycle(small, _Stub(), 10, 6, 60)
