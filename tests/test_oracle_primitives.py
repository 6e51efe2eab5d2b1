"""Pins of the oracle's building blocks against closed forms, hand values and
independent library routines (CPU only)."""

import math

import numpy as np
import pytest
import scipy.special
import torch
import torch.nn.functional as F

from oracle import model as om
from oracle.verify import ancestor_matrix, tree_attention
from tests.harness import micro_shape

rng = np.random.default_rng(1234)


# ---------------------------------------------------------------- RMSNorm ----

def test_rmsnorm_hand_value():
    # mean of squares of (3, 4) is 12.5; with eps = 1 the divisor is sqrt(13.5)
    out = om.rmsnorm(np.array([3.0, 4.0]), np.array([1.0, 2.0]), 1.0)
    d = math.sqrt(13.5)
    np.testing.assert_allclose(out, [3.0 / d, 8.0 / d], rtol=0, atol=1e-15)


def test_rmsnorm_matches_torch():
    x = rng.normal(size=(7, 33)) * 3
    g = rng.normal(size=33)
    ref = F.rms_norm(torch.from_numpy(x), (33,), torch.from_numpy(g), eps=1e-5).numpy()
    np.testing.assert_allclose(om.rmsnorm(x, g, 1e-5), ref, rtol=1e-13, atol=1e-13)


# ------------------------------------------------------------------- RoPE ----

def test_rope_inverse_frequencies_hand_values():
    np.testing.assert_allclose(om.rope_inv_freq(4, 10000.0), [1.0, 0.01], rtol=1e-15)
    np.testing.assert_allclose(om.rope_inv_freq(8, 500000.0),
                               [1.0, 500000.0 ** -0.25, 500000.0 ** -0.5, 500000.0 ** -0.75], rtol=1e-14)


def test_rope_matches_complex_rotation():
    # rotate-half pairing: element j pairs with j + dh/2 as (real, imaginary)
    # parts, and is multiplied by exp(i * pos * inv_freq_j)
    dh, base = 16, 10000.0
    x = rng.normal(size=(5, dh))
    pos = np.array([0, 1, 7, 300, 16383])
    z = x[:, : dh // 2] + 1j * x[:, dh // 2:]
    z = z * np.exp(1j * pos[:, None] * om.rope_inv_freq(dh, base)[None, :])
    ref = np.concatenate([z.real, z.imag], axis=1)
    np.testing.assert_allclose(om.rope(x, pos, base), ref, rtol=1e-13, atol=1e-13)


def test_rope_position_zero_is_identity_and_norm_preserving():
    x = rng.normal(size=(3, 4, 32))
    np.testing.assert_array_equal(om.rope(x, 0, 10000.0), x)
    y = om.rope(x, 12345, 500000.0)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)


def test_rope_scores_depend_only_on_relative_position():
    q, k = rng.normal(size=64), rng.normal(size=64)
    base = 500000.0
    a = om.rope(q, 10, base) @ om.rope(k, 3, base)
    b = om.rope(q, 1010, base) @ om.rope(k, 1003, base)
    c = om.rope(q, 11, base) @ om.rope(k, 3, base)
    assert abs(a - b) < 1e-11
    assert abs(a - c) > 1e-6


# ------------------------------------------------------- softmax and SiLU ----

def test_softmax_two_element_closed_form_and_scipy():
    s = np.array([0.0, math.log(3.0)])
    np.testing.assert_allclose(om.softmax(s), [0.25, 0.75], rtol=1e-15)
    x = rng.normal(size=(4, 9)) * 20
    np.testing.assert_allclose(om.softmax(x), scipy.special.softmax(x, axis=-1), rtol=1e-13)


def test_silu_matches_torch():
    z = np.linspace(-30, 30, 101)
    np.testing.assert_allclose(om.silu(z), F.silu(torch.from_numpy(z)).numpy(), rtol=1e-14, atol=1e-300)
    assert om.silu(np.array(0.0)) == 0.0


# ----------------------------------------------------------------- SwiGLU ----

def test_swiglu_hand_value_gate_first():
    # d = F = 1: gate weight 1, up weight 3, down weight 0.5, input 2
    # silu(2) * 6 * 0.5; swapping gate and up would give silu(6) * 2 * 0.5
    out = om.swiglu(np.array([[2.0]]), np.array([[1.0], [3.0]]), np.array([[0.5]]))
    want = 2.0 / (1.0 + math.exp(-2.0)) * 6.0 * 0.5
    assert abs(out[0, 0] - want) < 1e-14


def test_split_qkv_row_order():
    # rows of w_qkv: all query heads, then key heads, then value heads
    m = micro_shape(d_model=4, n_q_heads=2, n_kv_heads=1, head_dim=2)
    w = np.zeros((m.qkv_rows, 4))
    for r in range(m.qkv_rows):
        w[r, 0] = r
    q, k, v = om.split_qkv(np.array([[1.0, 0, 0, 0]]), w, m)
    np.testing.assert_array_equal(q[0], [[0, 1], [2, 3]])
    np.testing.assert_array_equal(k[0], [[4, 5]])
    np.testing.assert_array_equal(v[0], [[6, 7]])


# -------------------------------------------------------------------- MoE ----

def test_moe_identical_experts_reduce_to_dense():
    d, f, E = 8, 12, 5
    gu = rng.normal(size=(2 * f, d))
    dn = rng.normal(size=(d, f))
    L = {"w_router": rng.normal(size=(E, d)), "w_gate_up": np.stack([gu] * E),
         "w_down": np.stack([dn] * E)}
    h = rng.normal(size=(6, d))
    out, _ = om.moe(h, L, 2)
    np.testing.assert_allclose(out, om.swiglu(h, gu, dn), rtol=1e-12, atol=1e-12)


def test_moe_hand_example_top2_renormalised():
    # three experts, scalar model; router logits (0, ln 2, ln 5) -> p = (1, 2, 5)/8;
    # top-2 keeps experts 2 and 1 with weights 5/7 and 2/7
    d, f = 1, 1
    L = {"w_router": np.array([[0.0], [math.log(2.0)], [math.log(5.0)]]),
         "w_gate_up": np.array([[[1.0], [1.0]], [[1.0], [2.0]], [[1.0], [3.0]]]),
         "w_down": np.array([[[1.0]], [[1.0]], [[1.0]]])}
    h = np.array([[1.0]])
    out, _ = om.moe(h, L, 2)
    s1 = 1.0 / (1.0 + math.exp(-1.0))
    want = 5.0 / 7.0 * s1 * 3.0 + 2.0 / 7.0 * s1 * 2.0
    assert abs(out[0, 0] - want) < 1e-14


def test_moe_route_ties_go_to_lower_id():
    d = 2
    wr = np.array([[1.0, 0], [0.0, 0], [1.0, 0], [1.0, 0]])
    ids, wts, _ = om.moe_route(np.array([[1.0, 0.0]]), wr, 2)
    assert list(ids[0]) == [0, 2]
    np.testing.assert_allclose(wts[0], [0.5, 0.5])


# -------------------------------------------------------------- attention ----

def test_ancestor_matrix_hand_tree():
    parents = np.array([-1, 0, 0, 1, 3, 2])
    vis = ancestor_matrix(parents)
    want = {0: {0}, 1: {0, 1}, 2: {0, 2}, 3: {0, 1, 3}, 4: {0, 1, 3, 4}, 5: {0, 2, 5}}
    for i, s in want.items():
        assert set(np.nonzero(vis[i])[0]) == s


@pytest.mark.parametrize("hq,hkv", [(4, 4), (8, 2), (6, 3)])
def test_tree_attention_matches_torch_sdpa(hq, hkv):
    T, P, dh = 9, 13, 16
    parents = np.array([-1, 0, 0, 1, 1, 2, 4, 6, 6])
    vis = np.concatenate([np.ones((T, P), bool), ancestor_matrix(parents)], axis=1)
    q = rng.normal(size=(T, hq, dh))
    k, v = rng.normal(size=(T, hkv, dh)), rng.normal(size=(T, hkv, dh))
    Kp, Vp = rng.normal(size=(hkv, P, dh)), rng.normal(size=(hkv, P, dh))
    o = tree_attention(q, k, v, Kp, Vp, vis)
    # library routine: keys = prefix then tree slots, boolean mask, GQA by head repeat
    keys = np.concatenate([Kp, k.transpose(1, 0, 2)], axis=1)     # [Hkv, P+T, dh]
    vals = np.concatenate([Vp, v.transpose(1, 0, 2)], axis=1)
    rep = hq // hkv
    tq = torch.from_numpy(q.transpose(1, 0, 2).copy())
    tk = torch.from_numpy(np.repeat(keys, rep, axis=0))
    tv = torch.from_numpy(np.repeat(vals, rep, axis=0))
    ref = F.scaled_dot_product_attention(tq, tk, tv, attn_mask=torch.from_numpy(vis))
    np.testing.assert_allclose(o, ref.numpy().transpose(1, 0, 2), rtol=1e-12, atol=1e-12)


def test_tree_attention_empty_prefix_root_returns_own_value():
    # with no prefix the root can only see itself: its output is its own value
    T, dh = 3, 8
    parents = np.array([-1, 0, 1])
    vis = ancestor_matrix(parents)
    q, k, v = rng.normal(size=(T, 2, dh)), rng.normal(size=(T, 1, dh)), rng.normal(size=(T, 1, dh))
    o = tree_attention(q, k, v, np.zeros((1, 0, dh)), np.zeros((1, 0, dh)), vis)
    np.testing.assert_array_equal(o[0, 0], v[0, 0])
    np.testing.assert_array_equal(o[0, 1], v[0, 0])
