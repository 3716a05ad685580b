"""CPU oracle for the AdaPLD draft-and-verify step (test infrastructure only).

Only the tests, the package smoke check and the benchmark's CPU-baseline leg
may import this package.  It shares no code with the HIP path.
"""
from .adapld_oracle import (  # noqa: F401
    KIND_NONE, KIND_LEX, KIND_SEM, bf16_bits_to_f64, lexical_match, cosine_rows,
    semantic_topk, embedding_fallback, build_draft_tree, build_draft_tree_paper, tree_verify_attn, accept_greedy, compact_kv, step,
)
