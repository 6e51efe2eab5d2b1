"""Model shapes and verify workloads.

The target families are the ones the paper evaluates (Sec. 5: LLaMA2-Chat
7B/13B, LLaMA3-Instruct 8B/70B, Vicuna 7B, Qwen2 7B, Mixtral-8x7B).  The draft
tree follows the paper's appendix "Draft Tree Structure": 60 draft tokens at
depth 6; the per-depth widths of its dynamic tree are not published, so the
workloads use fixed widths.  Weights are random-init (no trained checkpoints
are available) and every workload is fully determined by its seeds.

Where the named public model fixes a hyper-parameter that the workload text
leaves open (RMSNorm epsilon, RoPE base), the public model's value is used.
"""

from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Dict, Tuple


@dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    n_experts: int = 1          # 1 = dense SwiGLU MLP
    top_k: int = 1              # experts per token (MoE only)
    rms_eps: float = 1e-5
    rope_base: float = 10000.0
    weight_std: float = 0.02    # std of every matrix and embedding entry
    gain_std: float = 0.1       # RMSNorm gains are 1 + N(0, gain_std^2), different per layer and norm

    @property
    def qkv_rows(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    def weight_bytes(self, experts_touched: int | None = None) -> int:
        """bf16 bytes of every weight a full verify pass reads."""
        d, f = self.d_model, self.d_ff
        e = self.n_experts if experts_touched is None else experts_touched
        per_layer = 2 * d  # two norm gains
        per_layer += self.qkv_rows * d + d * self.n_q_heads * self.head_dim
        if self.n_experts == 1:
            per_layer += 3 * f * d
        else:
            per_layer += e * 3 * f * d + self.n_experts * d
        total = self.n_layers * per_layer + self.vocab * d + d  # lm head + final norm
        return 2 * total

    def kv_bytes_per_position(self) -> int:
        """bf16 K+V bytes one cache position holds over all layers."""
        return 2 * 2 * self.n_layers * self.n_kv_heads * self.head_dim


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    batch: int
    prefix_len: int
    widths: Tuple[int, ...]      # draft nodes per depth (root excluded)
    plant: str                    # "leaf": plant a full root-to-leaf path; "half": Bernoulli(1/2), length U{0..D}
    kv_source: str                # "prefill": fp64 prefill of the random prefix; "synthetic": seeded i.i.d. K/V
    weight_seed: int = 0
    prefix_seed: int = 1
    tree_seed: int = 1000
    n_trees: int = 16
    description: str = ""
    max_tree: int = 64                                # node rows reserved per sequence
    prefix_lens: Tuple[int, ...] = ()                 # ragged batch: per-sequence prefix (else prefix_len)
    seq_widths: Tuple[Tuple[int, ...], ...] = ()      # ragged batch: per-sequence widths (else widths)

    def prefix_of(self, seq: int) -> int:
        return self.prefix_lens[seq] if self.prefix_lens else self.prefix_len

    def widths_of(self, seq: int) -> Tuple[int, ...]:
        return self.seq_widths[seq] if self.seq_widths else self.widths

    def prefixes(self):
        return [self.prefix_of(b) for b in range(self.batch)]

    @property
    def n_draft(self) -> int:
        """Draft nodes of the largest tree of the batch."""
        return max(int(sum(self.widths_of(b))) for b in range(self.batch))

    @property
    def tree_nodes(self) -> int:
        """Nodes per tree including the root (the largest tree of the batch)."""
        return 1 + self.n_draft

    @property
    def depth(self) -> int:
        return max(len(self.widths_of(b)) for b in range(self.batch))

    def kv_capacity(self, align: int = 64) -> int:
        need = max(self.prefixes()) + self.tree_nodes
        return ((need + align - 1) // align) * align


TINY = ModelShape("tiny", n_layers=2, d_model=256, n_q_heads=4, n_kv_heads=4, head_dim=64,
                  d_ff=688, vocab=1024, rms_eps=1e-6, rope_base=10000.0)
LLAMA2_7B = ModelShape("llama2-7b", n_layers=32, d_model=4096, n_q_heads=32, n_kv_heads=32,
                       head_dim=128, d_ff=11008, vocab=32000, rms_eps=1e-5, rope_base=10000.0)
LLAMA3_8B = ModelShape("llama3-8b", n_layers=32, d_model=4096, n_q_heads=32, n_kv_heads=8,
                       head_dim=128, d_ff=14336, vocab=128256, rms_eps=1e-5, rope_base=500000.0)
MIXTRAL_8X7B = ModelShape("mixtral-8x7b", n_layers=32, d_model=4096, n_q_heads=32, n_kv_heads=8,
                          head_dim=128, d_ff=14336, vocab=32000, n_experts=8, top_k=2,
                          rms_eps=1e-5, rope_base=1000000.0)

# Small shapes used only by parity tests: they exercise head_dim 128, GQA,
# MoE, ragged vocab / d_ff tails and several GEMM tiles while the fp64 oracle
# still finishes in seconds.
SMALL_GQA = ModelShape("small-gqa", n_layers=2, d_model=512, n_q_heads=8, n_kv_heads=2,
                       head_dim=128, d_ff=1376, vocab=3000, rms_eps=1e-5, rope_base=500000.0)
SMALL_MOE = ModelShape("small-moe", n_layers=2, d_model=512, n_q_heads=8, n_kv_heads=2,
                       head_dim=128, d_ff=704, vocab=2056, n_experts=8, top_k=2,
                       rms_eps=1e-5, rope_base=1000000.0)
SMALL_MHA = ModelShape("small-mha", n_layers=3, d_model=384, n_q_heads=3, n_kv_heads=3,
                       head_dim=128, d_ff=1000, vocab=4104, rms_eps=1e-5, rope_base=10000.0)

D6 = (10, 10, 10, 10, 10, 10)


def ragged_prefixes(batch: int, lo: int, hi: int, seed: int) -> Tuple[int, ...]:
    """Per-sequence prefix lengths spread uniformly over [lo, hi] (a serving
    batch of conversations at different points)."""
    import numpy as np
    rng = np.random.default_rng(seed)
    return tuple(int(x) for x in rng.integers(lo, hi + 1, size=batch))


def _chain2(batch: int) -> "Workload":
    return Workload(f"llama3-8b-chain2-b{batch}", LLAMA3_8B, batch=batch, prefix_len=2048, widths=(1, 1),
                    plant="half", kv_source="synthetic", max_tree=3,
                    prefix_lens=ragged_prefixes(batch, 256, 2048, 4242 + batch),
                    description=f"Llama-3-8B shape, B{batch}, ragged prefixes in [256, 2048], "
                                "a chain of 2 drafts per sequence")

WORKLOADS: Dict[str, Workload] = {
    w.name: w for w in [
        Workload("tiny", TINY, batch=1, prefix_len=128, widths=(2, 4, 4, 5), plant="leaf",
                 kv_source="prefill",
                 description="2L d256 4x64 MHA F688 V1024, P128, tree 15 nodes depth 4"),
        Workload("llama2-7b", LLAMA2_7B, batch=1, prefix_len=1024, widths=D6, plant="half",
                 kv_source="synthetic",
                 description="Llama-2-7B shape, bf16, B1, P1024, tree 60 nodes depth 6"),
        Workload("llama3-8b", LLAMA3_8B, batch=1, prefix_len=2048, widths=D6, plant="half",
                 kv_source="synthetic",
                 description="Llama-3-8B shape (GQA 32/8), bf16, B1, P2048, tree 60 nodes depth 6"),
        Workload("mixtral-8x7b", MIXTRAL_8X7B, batch=1, prefix_len=2048, widths=D6, plant="half",
                 kv_source="synthetic",
                 description="Mixtral-8x7B shape (8 experts top-2), bf16, B1, P2048, tree 60/6"),
        Workload("llama3-8b-longctx", LLAMA3_8B, batch=8, prefix_len=16384, widths=D6, plant="half",
                 kv_source="synthetic",
                 description="Llama-3-8B shape, B8 x P16384, one 60/6 tree per sequence"),
        # parity-test workloads (oracle-sized)
        Workload("small-gqa", SMALL_GQA, batch=2, prefix_len=200, widths=(3, 5, 8, 8, 6, 5),
                 plant="leaf", kv_source="prefill",
                 description="2L d512 GQA 8/2x128 F1376 V3000, B2, P200, tree 35/6"),
        Workload("small-moe", SMALL_MOE, batch=1, prefix_len=96, widths=D6, plant="leaf",
                 kv_source="prefill",
                 description="2L d512 GQA 8/2x128, 8 experts top-2 F704, V2056, P96, tree 60/6"),
        Workload("small-mha", SMALL_MHA, batch=3, prefix_len=70, widths=(4, 6, 6, 6, 4, 2),
                 plant="leaf", kv_source="prefill",
                 description="3L d384 MHA 3x128 F1000 V4104, B3, P70, tree 28/6"),
        # ragged serving batch: chains of 0-2 drafts, prefixes of different lengths
        Workload("small-chain2", SMALL_GQA, batch=16, prefix_len=200, widths=(1, 1), plant="half",
                 kv_source="prefill", max_tree=3, prefix_lens=ragged_prefixes(16, 20, 200, 77),
                 seq_widths=tuple((1, 1) if b % 5 else ((1,) if b % 10 else ()) for b in range(16)),
                 description="small-gqa model, B16, ragged prefixes in [20, 200], chains of 2 drafts "
                             "(sequences 5 and 15: 1, sequences 0 and 10: the root alone)"),
        *[_chain2(b) for b in (2, 4, 8, 16)],
    ]
}


@dataclass(frozen=True)
class DraftShape:
    """A GRIFFIN-style draft model for a target: Token-Guided Fusion (a 2d -> d
    fusion, a 2d -> tgf_dim up projection, a tgf_dim -> d down projection),
    one decoder layer of the target's shape, and the Token-Enhanced Head (two
    d x d heads); it shares the target's embedding, final norm and LM head.
    Expansion: `k` candidates per node and per depth, `depth` draft passes,
    `n_total` draft tokens kept."""
    target: ModelShape
    tgf_dim: int
    ln_eps: float = 1e-5
    k: int = 10
    depth: int = 6
    n_total: int = 60

    @property
    def layer(self) -> ModelShape:
        """The decoder layer as a one-layer model of the target's shape, with a
        dense SwiGLU MLP of the target's (expert) width also for MoE targets."""
        return replace(self.target, name=self.target.name + "-draft", n_layers=1, n_experts=1, top_k=1)

    def param_count(self) -> int:
        m, d, e = self.target, self.target.d_model, self.tgf_dim
        tgf = 2 * d * d + d + 4 * d + 2 * d * e + e + e * d + d
        layer = 2 * d + m.qkv_rows * d + d * m.n_q_heads * m.head_dim + 3 * d * m.d_ff
        teh = 2 * (d * d + d)
        return tgf + layer + teh


DRAFTS: Dict[str, DraftShape] = {
    # the expansion dimension is the value the paper's appendix gives (11008);
    # with it the draft of the 8B target has 0.42B parameters, as published
    "llama3-8b": DraftShape(LLAMA3_8B, tgf_dim=11008),
    "tiny": DraftShape(TINY, tgf_dim=1000, k=4, depth=4, n_total=12),
    "small-gqa": DraftShape(SMALL_GQA, tgf_dim=1800, k=5, depth=5, n_total=20),
    # vocabularies of several top-k slices (8192 logits each): one not a
    # multiple of 4 (scalar loads), one with 16-byte loads and the largest k
    # an MoE target: the draft's decoder layer is dense (expert width)
    "small-moe": DraftShape(SMALL_MOE, tgf_dim=900, k=4, depth=4, n_total=12),
    "tiny-v20001": DraftShape(replace(TINY, name="tiny-v20001", vocab=20001), tgf_dim=1000, k=4, depth=4,
                              n_total=12),
    "tiny-v20000": DraftShape(replace(TINY, name="tiny-v20000", vocab=20000), tgf_dim=1000, k=16, depth=3,
                              n_total=40),
}


def get_workload(name: str) -> Workload:
    try:
        return WORKLOADS[name]
    except KeyError as e:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(WORKLOADS)}") from e


def with_layers(w: Workload, n_layers: int) -> Workload:
    """Same workload with fewer layers (used for bounded CPU timing samples)."""
    return replace(w, model=replace(w.model, n_layers=n_layers))
