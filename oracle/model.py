"""Decoder building blocks of the target models, in fp64.

The paper (Sec. 5) evaluates LLaMA2/LLaMA3/Vicuna/Qwen2 decoders and Mixtral;
it does not restate their layers, so each block below is the standard public
definition of those families:

* RMSNorm: x / sqrt(mean(x^2) + eps) * g.
* Rotary embedding, "rotate-half" pairing (element j with j + dh/2),
  inverse frequency base^(-2j/dh), angle = position * inverse frequency.
* Grouped-query attention with contiguous groups: query head h reads KV head
  h // (Hq / Hkv); scores scaled by 1/sqrt(dh); softmax; no bias.
* SwiGLU MLP: (silu(h Wg^T) * (h Wu^T)) Wd^T, silu(z) = z / (1 + e^-z).
* Mixtral MoE: router logits h Wr^T, softmax over experts, keep the top-k
  (ties to the lower expert id), renormalise the kept probabilities, sum the
  kept experts' SwiGLU outputs weighted by them.

All weights are bf16 bit patterns upcast exactly to fp64.
"""

from __future__ import annotations

from typing import Dict, Optional

import numpy as np
import torch


def to_f64(t: Optional[torch.Tensor]) -> Optional[np.ndarray]:
    if t is None:
        return None
    return t.detach().to("cpu").to(torch.float64).numpy()


class OracleWeights:
    """fp64 view of a ``workloads.gen.ModelWeights``.

    With ``cache=True`` every upcast layer is kept; otherwise layers are upcast
    on each access (for shapes whose fp64 copy does not fit in host memory)."""

    def __init__(self, mw, cache: bool = True):
        self.mw = mw
        self.shape = mw.shape
        self.cache = cache
        self._layers: Dict[int, Dict[str, Optional[np.ndarray]]] = {}
        self._lm = None
        self.final_norm = to_f64(mw.final_norm)

    def embed(self, tokens) -> np.ndarray:
        idx = torch.as_tensor(np.asarray(tokens, dtype=np.int64))
        return to_f64(self.mw.embed.to("cpu")[idx])

    def layer(self, l: int) -> Dict[str, Optional[np.ndarray]]:
        if l in self._layers:
            return self._layers[l]
        L = {k: to_f64(v) for k, v in self.mw.layers[l].items()}
        if self.cache:
            self._layers[l] = L
        return L

    def lm_head(self) -> np.ndarray:
        if self._lm is not None:
            return self._lm
        lm = to_f64(self.mw.lm_head)
        if self.cache:
            self._lm = lm
        return lm


# ------------------------------------------------------------- primitives ----

def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope_inv_freq(dh: int, base: float) -> np.ndarray:
    j = np.arange(dh // 2, dtype=np.float64)
    return base ** (-2.0 * j / dh)


def rope(x: np.ndarray, pos, base: float) -> np.ndarray:
    """Rotate x[..., dh] at integer positions pos (broadcast over leading dims).

    pos has the shape of x without its last axis, or is broadcastable to it."""
    dh = x.shape[-1]
    half = dh // 2
    ang = np.asarray(pos, dtype=np.float64)[..., None] * rope_inv_freq(dh, base)
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def softmax(s: np.ndarray, axis: int = -1) -> np.ndarray:
    m = np.max(s, axis=axis, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=axis, keepdims=True)


def split_qkv(h: np.ndarray, w_qkv: np.ndarray, m):
    """h [n, d] -> q [n, Hq, dh], k [n, Hkv, dh], v [n, Hkv, dh] (no rotation)."""
    Hq, Hkv, dh = m.n_q_heads, m.n_kv_heads, m.head_dim
    y = h @ w_qkv.T
    q = y[:, : Hq * dh].reshape(-1, Hq, dh)
    k = y[:, Hq * dh: (Hq + Hkv) * dh].reshape(-1, Hkv, dh)
    v = y[:, (Hq + Hkv) * dh:].reshape(-1, Hkv, dh)
    return q, k, v


def swiglu(h: np.ndarray, w_gate_up: np.ndarray, w_down: np.ndarray) -> np.ndarray:
    f = w_down.shape[1]
    gate = h @ w_gate_up[:f].T
    up = h @ w_gate_up[f:].T
    return (silu(gate) * up) @ w_down.T


def moe_route(h: np.ndarray, w_router: np.ndarray, top_k: int):
    """Per row: kept expert ids (descending probability, ties to the lower id),
    their renormalised weights, and the router logits."""
    logits = h @ w_router.T                      # [n, E]
    p = softmax(logits, axis=-1)
    n, E = p.shape
    ids = np.zeros((n, top_k), dtype=np.int64)
    wts = np.zeros((n, top_k))
    for r in range(n):
        # stable sort on -p keeps the lower id first among equal probabilities
        order = np.argsort(-p[r], kind="stable")[:top_k]
        ids[r] = order
        wts[r] = p[r, order] / np.sum(p[r, order])
    return ids, wts, logits


def moe(h: np.ndarray, L: Dict[str, np.ndarray], top_k: int):
    """Each row gets the weighted sum of its kept experts' SwiGLU outputs,
    added in rank order (highest probability first).  Every expert's SwiGLU is
    evaluated once over all rows that keep it (rows are independent)."""
    ids, wts, logits = moe_route(h, L["w_router"], top_k)
    y = {}
    for e in sorted(set(int(x) for x in ids.ravel())):
        rows = np.nonzero((ids == e).any(axis=1))[0]
        y[e] = dict(zip(rows.tolist(), swiglu(h[rows], L["w_gate_up"][e], L["w_down"][e])))
    out = np.zeros_like(h)
    for r in range(h.shape[0]):
        for j in range(top_k):
            out[r] += wts[r, j] * y[int(ids[r, j])][r]
    return out, logits


def mlp(h: np.ndarray, L: Dict[str, np.ndarray], m):
    """Returns (mlp output, router logits or None)."""
    if m.n_experts == 1:
        return swiglu(h, L["w_gate_up"], L["w_down"]), None
    return moe(h, L, m.top_k)
