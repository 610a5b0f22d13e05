"""Oracle for the DSI verification step -- TEST INFRASTRUCTURE ONLY.

A plain, slow, fp64 CPU statement of what the verification step computes:
the target forward over a window of k drafted tokens against a cached prefix
(``forward64``) and the lossless accept/reject of those drafts (``verify64``),
plus exact enumerations that pin the accept/reject rule (``bruteforce``), and
the drafter side of a speculative-inference iteration with the loop built
from both (``drafting``: ``draft64``, ``si_loop64``).

Only the tests, the smoke check and the CPU-baseline leg of the benchmark may
import this package.  It shares no code with the HIP path and imports nothing
from it; the product path never calls it.

Parity status of each function (what pins it) is listed in its docstring.
Architecture choices of the forward (RMSNorm, rotate-half RoPE, GQA head
grouping, SwiGLU, untied head) are not fixed by the paper, which treats the
target LM as a black box (Appendix B); they are pinned by invariants, textbook
special cases and, for the whole decoder, by an independent implementation of
the same architecture (the transformers library's Llama model, loaded with
the same weights, in a CPU test).
"""
from .model import (bf16_round64, rmsnorm64, rope64, attention64, silu64,
                        layer64, head64, forward64, embed64)
from .verification import VerifyResult, softmax64, verify64
from . import bruteforce
from .drafting import DraftResult, draft64, draft_q32, draw_inverse_cdf, si_loop64
from .tree import ancestors, greedy64, tree_logits64, tree_walk, validate_tree

__all__ = [
    "bf16_round64", "rmsnorm64", "rope64", "attention64", "silu64", "layer64",
    "head64", "forward64", "embed64", "VerifyResult", "softmax64", "verify64",
    "bruteforce", "DraftResult", "draft64", "draft_q32", "draw_inverse_cdf",
    "si_loop64", "ancestors", "greedy64", "tree_logits64", "tree_walk", "validate_tree",
]
