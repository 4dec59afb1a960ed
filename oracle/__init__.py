"""CPU oracle for the unified AI-query pipeline -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct numpy implementation (fp64 for floating
point) of what the device pipeline computes, written from the paper's
definitions: the SQL-clause-to-tensor mapping of Table 1 (FROM -> input
arrays, WHERE -> boolean mask, AI_IF -> causal-LM classification on the
last position's Yes/No logits, SUM -> masked reduction) and the unified
classification program of Figure 2 (Section 3.1).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg
may import this package.  The product path (the HIP library and its Python
binding) never imports, links or calls anything here, and this package
imports nothing from the product path: the two share only the seeded input
generators of ``synth``.

Parity status: the paper prints no worked example with numeric values, so
no function here is pinned to a value printed in the paper; every function
is pinned instead by brute force on tiny inputs, closed forms, invariants or
an independent library formulation (see ``tests/test_oracle_*.py``).
"""
from .relational import (eval_pred, select, hash_join, sequences, pack, group_avg_count,
                         count_by)
from .transformer import (rmsnorm, rope, causal_attention, gelu_erf, silu, forward_hidden,
                          label_logits, full_logits, Weights64)
from .query import run_query, decide, aggregate, relational
from .pairs import candidate_pairs, pair_sequences
from .generate import position_logits, greedy_generate, generated_length, like_tokens

__all__ = [
    "eval_pred", "select", "hash_join", "sequences", "pack", "group_avg_count", "count_by",
    "rmsnorm", "rope", "causal_attention", "gelu_erf", "silu", "forward_hidden",
    "label_logits", "full_logits", "Weights64", "run_query", "decide", "aggregate", "relational",
    "position_logits", "greedy_generate", "generated_length", "like_tokens",
    "candidate_pairs", "pair_sequences",
]
