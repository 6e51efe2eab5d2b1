"""Python binding of the tree-verification library (argument marshalling only).

Every step of the verify pass runs in the HIP library; PyTorch only owns device
memory (weights, KV cache, optional logits) and provides the stream.
"""

from __future__ import annotations

import ctypes
from ctypes import POINTER, byref, c_float, c_int32, c_uint64, c_void_p
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np
import torch

from . import _native as N


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _p32(a: np.ndarray):
    return a.ctypes.data_as(POINTER(c_int32))


def _check(rc: int, what: str, ctx=None):
    if rc != N.GRIFFIN_OK:
        detail = ""
        if ctx is not None and ctx.value:
            detail = N.lib.griffin_last_error(ctx).decode()
        raise N.GriffinError(rc, what + (f" ({detail})" if detail else ""))


@dataclass
class AcceptResult:
    length: np.ndarray     # [B] accepted draft tokens L
    tokens: np.ndarray     # [B, max_depth + 1] L tokens then the target's next token, -1 padded
    path: np.ndarray       # [B, max_depth] accepted node ids, -1 padded
    status: int = 0        # GRIFFIN_OK or GRIFFIN_ENUMERIC

    def sequence(self, b: int):
        L = int(self.length[b])
        return L, [int(t) for t in self.tokens[b, : L + 1]], [int(n) for n in self.path[b, :L]]


def pack_trees(trees: Sequence, max_tree: int):
    """Lay out trees (objects with .tokens / .parents) as [B][max_tree] arrays."""
    B = len(trees)
    tok = np.zeros((B, max_tree), dtype=np.int32)
    par = np.full((B, max_tree), -1, dtype=np.int32)
    n = np.zeros(B, dtype=np.int32)
    for b, t in enumerate(trees):
        k = len(t.tokens)
        tok[b, :k] = t.tokens
        par[b, :k] = t.parents
        n[b] = k
    return n, tok, par


def tree_prepare(tokens, parents, prefix_len: int, max_tree: int, max_depth: int, vocab: int, kv_capacity: int):
    """Host-only validation + metadata (depth, position, ancestor masks) of one tree."""
    tok, par = _i32(tokens), _i32(parents)
    n = len(tok)
    depth = np.zeros(max(n, 1), dtype=np.int32)
    pos = np.zeros(max(n, 1), dtype=np.int32)
    anc = np.zeros(max(n, 1), dtype=np.uint64)
    rc = N.lib.griffin_tree_prepare(n, _p32(tok), _p32(par), prefix_len, max_tree, max_depth, vocab, kv_capacity,
                                    _p32(depth), _p32(pos), anc.ctypes.data_as(POINTER(c_uint64)))
    return rc, depth[:n], pos[:n], anc[:n]


def accept_walk(trees: Sequence, pred: np.ndarray, max_tree: int, max_depth: int, vocab: int,
                stream: Optional[torch.cuda.Stream] = None) -> AcceptResult:
    """Device acceptance walk on given per-node predictions pred [B][max_tree]."""
    n, tok, par = pack_trees(trees, max_tree)
    B = len(trees)
    pred = _i32(pred)
    L = np.zeros(B, dtype=np.int32)
    out = np.zeros((B, max_depth + 1), dtype=np.int32)
    path = np.zeros((B, max(max_depth, 1)), dtype=np.int32)
    s = (stream or torch.cuda.current_stream()).cuda_stream
    rc = N.lib.griffin_accept_walk(c_void_p(s), B, max_tree, max_depth, vocab, _p32(n), _p32(tok), _p32(par),
                                   _p32(pred), _p32(L), _p32(out), _p32(path))
    _check(rc, "griffin_accept_walk")
    return AcceptResult(L, out, path[:, :max_depth])


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32))


def _pf32(a: np.ndarray):
    return a.ctypes.data_as(POINTER(c_float))


def _device_rows(t: Optional[torch.Tensor], rows: int, vocab: int, what: str, optional: bool = False):
    if t is None and optional:
        return c_void_p(None)
    if t is None or not (t.is_cuda and t.dtype == torch.float32 and t.is_contiguous() and t.numel() >= rows * vocab):
        raise ValueError(f"{what} must be a contiguous fp32 CUDA tensor with [B*max_tree, vocab] elements")
    return c_void_p(t.data_ptr())


def accept_sampled_walk(trees: Sequence, logits: torch.Tensor, q_draft: Optional[torch.Tensor], u_accept, u_final,
                        temperature: float, max_tree: int, max_depth: int, vocab: int,
                        stream: Optional[torch.cuda.Stream] = None, noalloc: bool = False) -> AcceptResult:
    """Device stochastic acceptance (temperature > 0) on given logits and
    draft distributions, both fp32 [B*max_tree, vocab] CUDA tensors (q_draft
    None: a deterministic draft, each child a point mass at its token); the
    uniforms are [B, max_tree] arrays in [0, 1).  noalloc: the entry point
    that uses the library's fixed device block instead of allocating."""
    n, tok, par = pack_trees(trees, max_tree)
    B = len(trees)
    ua, uf = _f32(u_accept).reshape(B, max_tree), _f32(u_final).reshape(B, max_tree)
    L = np.zeros(B, dtype=np.int32)
    out = np.zeros((B, max_depth + 1), dtype=np.int32)
    path = np.zeros((B, max(max_depth, 1)), dtype=np.int32)
    s = (stream or torch.cuda.current_stream()).cuda_stream
    name = "griffin_accept_sampled_walk_noalloc" if noalloc else "griffin_accept_sampled_walk"
    rc = getattr(N.lib, name)(
        c_void_p(s), B, max_tree, max_depth, vocab, _p32(n), _p32(tok), _p32(par),
        _device_rows(logits, B * max_tree, vocab, "logits"),
        _device_rows(q_draft, B * max_tree, vocab, "q_draft", optional=True),
        _pf32(ua), _pf32(uf), float(temperature), _p32(L), _p32(out), _p32(path))
    _check(rc, name)
    return AcceptResult(L, out, path[:, :max_depth])


def write_prefix(k_cache: torch.Tensor, v_cache: torch.Tensor, shape, max_batch: int, kv_capacity: int, layer: int,
                 seq: int, k: torch.Tensor, v: torch.Tensor, stream) -> None:
    """Copy a prefix k, v bf16 [Hkv, P, dh] (k post-rotary) into the cache
    layouts of griffin_verify_init: K [layers][batch][Hkv][cap][dh], V in
    transposed 32-slot tiles [layers][batch][Hkv][cap / 32][dh][32]."""
    Hkv, dh = shape.n_kv_heads, shape.head_dim
    P = k.shape[1]
    full, rem = divmod(P, 32)
    tiles = v_cache.view(shape.n_layers, max_batch, Hkv, kv_capacity // 32, dh, 32)[layer, seq]
    stream.wait_stream(torch.cuda.current_stream(k.device))  # k, v may still be in flight on the caller's stream
    with torch.cuda.stream(stream):
        k_cache.view(shape.n_layers, max_batch, Hkv, kv_capacity, dh)[layer, seq, :, :P, :].copy_(k)
        if full:
            tiles[:, :full].copy_(v[:, : full * 32].reshape(v.shape[0], full, 32, v.shape[2]).transpose(-1, -2))
        if rem:
            tiles[:, full, :, :rem].copy_(v[:, full * 32:].transpose(-1, -2))


class TreeVerifier:
    """One verify context: borrowed weights, a KV cache, and the library's workspace.

    shape: object with n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ff,
           vocab, n_experts, top_k, rms_eps, rope_base.
    weights: object with embed, lm_head, final_norm (bf16 CUDA tensors) and
           layers[l] = dict(attn_norm, w_qkv, w_o, mlp_norm, w_gate_up, w_down, w_router).
    """

    def __init__(self, shape, weights, *, max_batch: int, max_tree: int, max_depth: int, kv_capacity: int,
                 k_cache: Optional[torch.Tensor] = None, v_cache: Optional[torch.Tensor] = None,
                 stream: Optional[torch.cuda.Stream] = None):
        self.shape = shape
        self.max_batch, self.max_tree, self.max_depth, self.kv_capacity = max_batch, max_tree, max_depth, kv_capacity
        self.desc = N.ModelDesc(shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                                shape.d_ff, shape.vocab, shape.n_experts, shape.top_k, shape.rms_eps,
                                shape.rope_base, max_batch, max_tree, max_depth, kv_capacity)
        dev = weights.embed.device
        if dev.type != "cuda":
            raise ValueError("weights must be device tensors")
        L, Hkv, dh = shape.n_layers, shape.n_kv_heads, shape.head_dim
        if k_cache is None:
            k_cache = torch.zeros((L, max_batch, Hkv, kv_capacity, dh), dtype=torch.bfloat16, device=dev)
        if v_cache is None:
            v_cache = torch.zeros((L, max_batch, Hkv, kv_capacity // 32, dh, 32), dtype=torch.bfloat16, device=dev)
        need = N.lib.griffin_kv_cache_bytes(byref(self.desc))
        for t in (k_cache, v_cache):
            if t.dtype != torch.bfloat16 or not t.is_contiguous() or t.numel() * 2 != need:
                raise ValueError("KV cache tensors must be contiguous bf16 of griffin_kv_cache_bytes bytes")
        self.k_cache, self.v_cache = k_cache, v_cache
        self.stream = stream or torch.cuda.current_stream(dev)
        self._weights = weights  # keep alive

        def arr(key):
            ptrs = [(lay[key].data_ptr() if lay.get(key) is not None else None) for lay in weights.layers]
            return (c_void_p * L)(*ptrs)

        self._arrays = {k: arr(k) for k in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")}
        self._arrays["w_router"] = arr("w_router") if shape.n_experts > 1 else None
        cast = lambda a: ctypes.cast(a, POINTER(c_void_p)) if a is not None else None  # noqa: E731
        self.w = N.Weights(weights.embed.data_ptr(), weights.lm_head.data_ptr(), weights.final_norm.data_ptr(),
                           cast(self._arrays["attn_norm"]), cast(self._arrays["w_qkv"]), cast(self._arrays["w_o"]),
                           cast(self._arrays["mlp_norm"]), cast(self._arrays["w_gate_up"]),
                           cast(self._arrays["w_down"]), cast(self._arrays["w_router"]))
        self.ctx = c_void_p()
        # init repacks the weights on the library's stream: order it after the
        # caller's stream, where the weights and caches were produced
        self.stream.wait_stream(torch.cuda.current_stream(dev))
        rc = N.lib.griffin_verify_init(byref(self.desc), byref(self.w), k_cache.data_ptr(), v_cache.data_ptr(),
                                       c_void_p(self.stream.cuda_stream), byref(self.ctx))
        _check(rc, "griffin_verify_init")
        self._batch = 0

    # ------------------------------------------------------------ KV cache ----
    def _v_tiles(self, layer: int, seq: int) -> torch.Tensor:
        Hkv, dh = self.shape.n_kv_heads, self.shape.head_dim
        return self.v_cache.view(self.shape.n_layers, self.max_batch, Hkv, self.kv_capacity // 32, dh, 32)[layer, seq]

    def write_prefix(self, layer: int, seq: int, k: torch.Tensor, v: torch.Tensor):
        """Place a cached prefix: k, v bf16 [Hkv, P, dh] (k post-rotary)."""
        write_prefix(self.k_cache, self.v_cache, self.shape, self.max_batch, self.kv_capacity, layer, seq, k, v,
                     self.stream)

    def read_v(self, layer: int, seq: int, n: int) -> torch.Tensor:
        """Cached values of slots [0, n) as [Hkv, n, dh]."""
        tiles = self._v_tiles(layer, seq)
        Hkv, nt, dh, _ = tiles.shape
        return tiles.transpose(-1, -2).reshape(Hkv, nt * 32, dh)[:, :n]

    # ---------------------------------------------------------------- step ----
    def step(self, prefix_len, trees: Sequence, logits_out: Optional[torch.Tensor] = None):
        n, tok, par = pack_trees(trees, self.max_tree)
        return self.step_arrays(prefix_len, n, tok, par, logits_out)

    def step_arrays(self, prefix_len, n_nodes, tokens, parents, logits_out: Optional[torch.Tensor] = None):
        B = len(n_nodes)
        pl, nn, tk, pa = _i32(prefix_len), _i32(n_nodes), _i32(tokens), _i32(parents)
        lp = None
        if logits_out is not None:
            if logits_out.dtype != torch.float32 or not logits_out.is_contiguous() or \
                    logits_out.numel() < B * self.max_tree * self.shape.vocab:
                raise ValueError("logits_out must be contiguous fp32 [B*max_tree, vocab]")
            lp = c_void_p(logits_out.data_ptr())
            # the caller may have touched the buffer on its own stream
            self.stream.wait_stream(torch.cuda.current_stream(logits_out.device))
        rc = N.lib.griffin_verify_step(self.ctx, B, _p32(pl), _p32(nn), _p32(tk), _p32(pa), lp)
        _check(rc, "griffin_verify_step", self.ctx)
        self._batch = B

    def accept(self, check: bool = True) -> AcceptResult:
        B, D = self._batch, self.max_depth
        L = np.zeros(max(B, 1), dtype=np.int32)
        out = np.zeros((max(B, 1), D + 1), dtype=np.int32)
        path = np.zeros((max(B, 1), max(D, 1)), dtype=np.int32)
        rc = N.lib.griffin_accept(self.ctx, _p32(L), _p32(out), _p32(path))
        if rc != N.CODES["GRIFFIN_ENUMERIC"] or check:
            _check(rc, "griffin_accept", self.ctx)
        return AcceptResult(L[:B], out[:B], path[:B, :D], rc)

    def accept_sampled(self, logits: torch.Tensor, q_draft: Optional[torch.Tensor], u_accept, u_final,
                       temperature: float = 1.0, check: bool = True) -> AcceptResult:
        """Stochastic acceptance (temperature > 0) of the last step: logits is
        the logits_out tensor that step filled, q_draft the draft distributions
        (fp32 [B*max_tree, vocab] CUDA tensor) or None for a deterministic
        draft such as DraftModel.tree's top-k expansion, u_accept / u_final
        uniforms [B, max_tree] in [0, 1)."""
        B, D, T = self._batch, self.max_depth, self.max_tree
        V = self.shape.vocab
        ua, uf = _f32(u_accept).reshape(B, T), _f32(u_final).reshape(B, T)
        L = np.zeros(max(B, 1), dtype=np.int32)
        out = np.zeros((max(B, 1), D + 1), dtype=np.int32)
        path = np.zeros((max(B, 1), max(D, 1)), dtype=np.int32)
        rc = N.lib.griffin_accept_sampled(self.ctx, _device_rows(logits, B * T, V, "logits"),
                                          _device_rows(q_draft, B * T, V, "q_draft", optional=True),
                                          _pf32(ua), _pf32(uf),
                                          float(temperature), _p32(L), _p32(out), _p32(path))
        if rc != N.CODES["GRIFFIN_ENUMERIC"] or check:
            _check(rc, "griffin_accept_sampled", self.ctx)
        return AcceptResult(L[:B], out[:B], path[:B, :D], rc)

    def predictions(self) -> np.ndarray:
        pred = np.zeros((max(self._batch, 1), self.max_tree), dtype=np.int32)
        rc = N.lib.griffin_read_predictions(self.ctx, _p32(pred))
        _check(rc, "griffin_read_predictions", self.ctx)
        return pred[: self._batch]

    def margins(self) -> np.ndarray:
        """Top-2 logit margin of every node of the last step: [batch, max_tree]
        fp32, -1 for absent nodes."""
        out = np.zeros((max(self._batch, 1), self.max_tree), dtype=np.float32)
        rc = N.lib.griffin_read_margins(self.ctx, _pf32(out))
        _check(rc, "griffin_read_margins", self.ctx)
        return out[: self._batch]

    def router_logits(self) -> np.ndarray:
        """MoE models: the fp32 router logits of the last step's pass,
        [n_layers, batch, max_tree, n_experts] (zeros for absent nodes)."""
        out = np.zeros((self.shape.n_layers, max(self._batch, 1), self.max_tree, self.shape.n_experts),
                       dtype=np.float32)
        rc = N.lib.griffin_read_router_logits(self.ctx, _pf32(out))
        _check(rc, "griffin_read_router_logits", self.ctx)
        return out[:, : self._batch]

    def set_bf16_activations(self, enable: bool):
        """GEMM activations as bf16 alone (True) or bf16 high + low parts
        (False, the default); see griffin_set_activation_precision."""
        rc = N.lib.griffin_set_activation_precision(self.ctx, 1 if enable else 0)
        _check(rc, "griffin_set_activation_precision", self.ctx)

    def features(self, nodes) -> torch.Tensor:
        """The target's features (hidden state after the last layer, before the
        final norm) of the last step's nodes: nodes[b] lists node ids of
        sequence b (all lists of one length; -1 gives a zero row).  Returns a
        CUDA float32 tensor [B, n, d_model], filled in stream order."""
        ids = np.asarray(nodes, dtype=np.int32)
        if ids.ndim != 2:
            raise ValueError("nodes must be a [batch][n] array")
        B, n = ids.shape
        out = torch.empty((B, n, self.shape.d_model), dtype=torch.float32, device=self.k_cache.device)
        ids = np.ascontiguousarray(ids)
        rc = N.lib.griffin_read_features(self.ctx, B, n, _p32(ids), c_void_p(out.data_ptr()))
        _check(rc, "griffin_read_features", self.ctx)
        return out

    def close(self):
        if getattr(self, "ctx", None) is not None and self.ctx.value:
            N.lib.griffin_verify_free(self.ctx)
            self.ctx = c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def _profile_enable(self, mask: int = (1 << len(N.KERNEL_CLASSES)) - 1):
    _check(N.lib.griffin_profile_enable(self.ctx, mask), "griffin_profile_enable", self.ctx)


def _profile_read(self) -> dict:
    """Per kernel class: (summed ms, launches) since the last read."""
    ms = (ctypes.c_double * len(N.KERNEL_CLASSES))()
    n = (ctypes.c_int64 * len(N.KERNEL_CLASSES))()
    _check(N.lib.griffin_profile_read(self.ctx, ms, n), "griffin_profile_read", self.ctx)
    return {name: (float(ms[k]), int(n[k])) for k, name in enumerate(N.KERNEL_CLASSES)}


def _set_graphs(self, enable: bool = True):
    """Replay each step's launch sequence from a captured HIP graph (default)
    or launch kernel by kernel."""
    _check(N.lib.griffin_set_graphs(self.ctx, 1 if enable else 0), "griffin_set_graphs", self.ctx)


TreeVerifier.profile_enable = _profile_enable
TreeVerifier.profile_read = _profile_read
def _commit(self):
    """Move the last step's accepted path into the KV cache (slots
    prefix_len + 1 .. prefix_len + L); continue with prefix_len + L + 1."""
    _check(N.lib.griffin_commit(self.ctx), "griffin_commit", self.ctx)


TreeVerifier.set_graphs = _set_graphs
TreeVerifier.commit = _commit
