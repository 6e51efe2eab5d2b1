"""Python binding of the draft model in the HIP library (griffin_draft_* in
include/griffin_verify.h): argument marshalling only."""

from __future__ import annotations

from ctypes import POINTER, byref, c_float, c_void_p
from typing import Optional, Sequence

import numpy as np
import torch

from . import _native as N
from .verifier import _check, _i32, _p32, pack_trees, write_prefix


def _pf(a: np.ndarray):
    return a.ctypes.data_as(POINTER(c_float))


class DraftModel:
    """A draft context: TGF, one decoder layer and the two heads, sharing the
    target's embedding, final norm and LM head.

    ds: DraftShape; weights: DraftWeights with CUDA tensors; target: the
    target's ModelWeights (CUDA; embed, lm_head, final_norm are used)."""

    def __init__(self, ds, weights, target, *, max_batch: int, max_tree: int, max_depth: int, kv_capacity: int,
                 stream: Optional[torch.cuda.Stream] = None):
        m = ds.layer
        self.ds, self.shape = ds, m
        self.max_batch, self.max_tree, self.max_depth, self.kv_capacity = max_batch, max_tree, max_depth, kv_capacity
        self.desc = N.ModelDesc(1, m.d_model, m.n_q_heads, m.n_kv_heads, m.head_dim, m.d_ff, m.vocab, 1, 1,
                                m.rms_eps, m.rope_base, max_batch, max_tree, max_depth, kv_capacity)
        dev = target.embed.device
        Hkv, dh = m.n_kv_heads, m.head_dim
        self.k_cache = torch.zeros((1, max_batch, Hkv, kv_capacity, dh), dtype=torch.bfloat16, device=dev)
        self.v_cache = torch.zeros((1, max_batch, Hkv, kv_capacity // 32, dh, 32), dtype=torch.bfloat16, device=dev)
        self.stream = stream or torch.cuda.current_stream(dev)
        self._keep = (weights, target)
        t, L = weights.t, weights.layer
        self.w = N.DraftWeights(*[t[n].data_ptr() for n in ("w_m", "b_m", "ln_h_g", "ln_h_b", "ln_x_g", "ln_x_b",
                                                            "w_u", "b_u", "w_d", "b_d", "w_p", "b_p", "w_r", "b_r")],
                                *[L[n].data_ptr() for n in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up",
                                                            "w_down")])
        self.h = c_void_p()
        rc = N.lib.griffin_draft_init(byref(self.desc), ds.tgf_dim, ds.ln_eps, byref(self.w),
                                      target.embed.data_ptr(), target.lm_head.data_ptr(),
                                      target.final_norm.data_ptr(), self.k_cache.data_ptr(),
                                      self.v_cache.data_ptr(), c_void_p(self.stream.cuda_stream), byref(self.h))
        _check(rc, "griffin_draft_init")

    def _ctx(self):
        return c_void_p(N.lib.griffin_draft_context(self.h))

    def write_prefix(self, seq: int, k: torch.Tensor, v: torch.Tensor):
        """The draft layer's cached prefix of sequence seq: k, v bf16 [Hkv, P, dh]."""
        write_prefix(self.k_cache, self.v_cache, self.shape, self.max_batch, self.kv_capacity, 0, seq, k, v,
                     self.stream)

    @staticmethod
    def _features(root_features: torch.Tensor, B: int, d: int):
        if (root_features.device.type != "cuda" or root_features.dtype != torch.float32
                or not root_features.is_contiguous() or tuple(root_features.shape) != (B, d)):
            raise ValueError(f"root_features must be a contiguous CUDA float32 tensor of shape {(B, d)}")
        return c_void_p(root_features.data_ptr())

    def step(self, prefix_len, trees: Sequence, root_features: torch.Tensor, k: int):
        """One draft pass; returns top-k tokens and log-probabilities [B, max_tree, k]."""
        n, tok, par = pack_trees(trees, self.max_tree)
        B = len(trees)
        P = _i32(prefix_len)
        ktok = np.zeros((B * self.max_tree, k), dtype=np.int32)
        klp = np.zeros((B * self.max_tree, k), dtype=np.float32)
        rc = N.lib.griffin_draft_step(self.h, B, _p32(P), _p32(n), _p32(tok), _p32(par),
                                      self._features(root_features, B, self.shape.d_model), k, _p32(ktok), _pf(klp))
        _check(rc, "griffin_draft_step", self._ctx())
        return ktok.reshape(B, self.max_tree, k), klp.reshape(B, self.max_tree, k)

    def extend(self, prefix_len, tokens: Sequence, features: torch.Tensor):
        """Write the draft layer's K/V of accepted tokens into its cache:
        tokens[b] (a list) at positions prefix_len[b] + j, features a CUDA
        float32 tensor [B, max_tree, d] whose row j is the target's feature of
        the token before tokens[b][j].  The caller continues with
        prefix_len[b] + len(tokens[b])."""
        B, T, d = len(tokens), self.max_tree, self.shape.d_model
        if (features.device.type != "cuda" or features.dtype != torch.float32 or not features.is_contiguous()
                or tuple(features.shape) != (B, T, d)):
            raise ValueError(f"features must be a contiguous CUDA float32 tensor of shape {(B, T, d)}")
        if not all(1 <= len(t) <= T for t in tokens):
            raise ValueError(f"every chain must hold 1 to {T} tokens")
        n = _i32([len(t) for t in tokens])
        tok = np.zeros((B, T), dtype=np.int32)
        for b, t in enumerate(tokens):
            tok[b, : len(t)] = t
        rc = N.lib.griffin_draft_extend(self.h, B, _p32(_i32(prefix_len)), _p32(n), _p32(tok),
                                        c_void_p(features.data_ptr()))
        _check(rc, "griffin_draft_extend", self._ctx())

    def tree(self, prefix_len, root_tokens, root_features: torch.Tensor, k: int, depth: int, n_total: int):
        """Draft one tree per sequence; returns (n_nodes [B], tokens, parents, scores [B, max_tree])."""
        B = len(root_tokens)
        P, roots = _i32(prefix_len), _i32(root_tokens)
        n = np.zeros(B, dtype=np.int32)
        tok = np.zeros((B, self.max_tree), dtype=np.int32)
        par = np.zeros((B, self.max_tree), dtype=np.int32)
        sc = np.zeros((B, self.max_tree), dtype=np.float32)
        rc = N.lib.griffin_draft_tree(self.h, B, _p32(P), _p32(roots), self._features(root_features, B,
                                      self.shape.d_model), k, depth, n_total, _p32(n), _p32(tok), _p32(par), _pf(sc))
        _check(rc, "griffin_draft_tree", self._ctx())
        return n, tok, par, sc

    def close(self):
        if getattr(self, "h", None) is not None and self.h.value:
            N.lib.griffin_draft_free(self.h)
            self.h = c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
