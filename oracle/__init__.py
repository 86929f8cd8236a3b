"""CPU oracle for DARTree draft-tree construction.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import or run anything in this package.
The product path (``paper_2608_13524_amd``) never imports it, and this package
imports nothing from the product path: the two share no code.
"""
from .dartree_ref import (  # noqa: F401
    BF16, FP32, Decoded, Level, Params, Supertree, Tree, build_supertree,
    build_tree, child_states, emit_batch, emit_tree, head_features,
    log_softmax, path_score, prepare, prune, rnd_bf16, select_level, topk_ids,
    vocab_logits,
)
