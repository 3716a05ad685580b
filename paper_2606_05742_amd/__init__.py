"""AdaPLD draft-and-verify hot path on MI355X (gfx950).

The four steps of one decoding iteration run as hand-written HIP kernels
behind the C-ABI library ``libadapld.so``; ``binding`` is a thin layer over
it (argument marshalling only).  A missing library is an error, never a
fallback.
"""
from .binding import (  # noqa: F401
    KIND_LEX, KIND_NONE, KIND_SEM, SUCC_EVERY_BRANCH, SUCC_SEMANTIC_ONLY, AdapldError, StepBuffers, accept_greedy, build_draft_tree, build_draft_tree_paper,
    NgramIndex, StepCall, lexical_match, load_library, semantic_topk, semantic_topk_embed, step, step_calls, tree_verify_attn,
    verify_plan, workspace_bytes,
)
