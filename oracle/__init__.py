"""CPU oracle for LLMCad's token-tree verification pass (arXiv 2309.04255, §3.2).

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, obviously correct
NumPy (float64) statement of what the verification pass computes.  Only the
test suite, the package entry's smoke check and the benchmark's CPU-baseline
leg may import it.  It shares no code with the HIP path: it imports neither
the library package nor its binding, and the library never imports it.

Contents
  model.py  the decoder forward as the plain causal definition, and the
            tree-masked forward over every node of a token tree
            (§3.2 "Tree decoder" masking table; "Batched non-autoregressive
            verification")
  walk.py   greedy acceptance: branch correct sequences, the correct token
            tree and its depth-first longest path (§3.2 "Depth-first verified
            sequence searching")
  decode.py greedy decoding, plainly and by the generate-and-verify loop
            with rollback of the token tree to its verified sequence (§3.1,
            §3.2 "Token tree verification and rectification")
  draft.py  draft-side tree generation: the tree decoder, the 30% branch
            threshold and the confidence-based branch pacer (§3.1, §3.2
            "Token tree generation", Eq. 1), with the fallback stop
  fallback.py  self-adaptive fallback: tree-cumulative confidence and the
            threshold update of Eq. 3 (§3.3)
  quant.py  group-wise 4-bit weights (the INT4 targets of §4.1): the
            dequantisation w = s (q - 8)

Every function is pinned by tests/test_oracle_*.py against something other
than itself: brute force, an independent library implementation
(transformers' LLaMA), closed forms, invariants or hand-built cases.  The
readings taken where the paper is silent or garbled are listed with the
build's design notes.
"""

from .model import (  # noqa: F401
    OracleConfig,
    OracleWeights,
    bf16_round,
    rmsnorm,
    rope,
    silu,
    causal_forward,
    prefill_kv,
    tree_forward,
    tree_layer,
    logits_from_stream,
    verify_tree,
)
from .walk import accept_walk, branch_sequences, correct_sequences  # noqa: F401
from .decode import commit_path, greedy_decode, speculative_decode  # noqa: F401
from .draft import generate_tree  # noqa: F401
from .fallback import DEFAULT_ALPHA, tree_confidence, update_alpha, most_matching_branch  # noqa: F401
from .quant import dequantize, unpack_codes  # noqa: F401
