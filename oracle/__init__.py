"""fp64 CPU oracle for GRIFFIN-style tree verification.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package: only the tests, the smoke check and the benchmark's CPU
baseline leg use it.  It shares no code with the HIP library; both sides only
consume the seeded inputs from the ``workloads`` package.

What it computes (the paper, Sec. 3 and Sec. 4.1): the target model scores
every draft token of a tree in one forward pass, and a draft token is kept only
if the target's own greedy prediction at its parent equals it; a rejected token
discards everything below it.  Sec. 5 runs the targets at temperature 0 (greedy)
and batch 1, and counts the acceptance length including the target's own next
token.  The target models are the LLaMA-family decoders and Mixtral named in
Sec. 5; their layer definitions (RMSNorm, rotary embedding, grouped-query
attention, SwiGLU MLP, softmax top-2 MoE) are written out plainly in
``model.py``.

Modules
  model.py    decoder building blocks in fp64
  verify.py   one tree-verification pass: all tree nodes, ancestor masks
  accept.py   greedy argmax and the acceptance walk (DFS, trie match)
  decode.py   plain causal decoding, fp64 prefill, greedy continuation,
              brute-force acceptance over root-to-leaf paths
  latency.py  the paper's speedup model (appendix on decoding latency)
  sampling.py stochastic tree acceptance at temperature T > 0 (Sec. 5)
  draft.py    the draft model's forward (TGF, decoder layer, TEH, Sec. 4.2)
              and the dynamic draft-tree expansion

Each function states which pins in ``tests/test_oracle_*.py`` hold it to the
paper or to mathematics it does not share with itself.  Absolute logits of a
random-init model have no published values: beyond those pins they are
"parity unpinned".
"""

from .model import OracleWeights  # noqa: F401
from .verify import verify_tree, VerifyResult  # noqa: F401
from .accept import argmax_first, top2_margin, accept_dfs, accept_trie  # noqa: F401
from .decode import DecodeCache, decode_step, prefill, greedy_chain, brute_force_accept  # noqa: F401
from .latency import speedup_ratio  # noqa: F401
from .sampling import softmax_t, draw, accept_sampled  # noqa: F401
from .draft import (DraftOracleWeights, DraftResult, Expansion, draft_forward, expand_tree, layernorm,  # noqa: F401
                    tgf, topk_logprobs)
