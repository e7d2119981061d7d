"""Plain fp64 CPU oracle of tree verification.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
link this package: only the tests, the package smoke check and the CPU
baseline leg of the benchmark use it.  It shares no code with the HIP path.

Contents
  tree_attention  -- tree-masked softmax attention with the full mask
                     materialised (Sec. 2.2, tree-causal mask and masked
                     attention equations).
  tree_accept     -- per-node target argmax and greedy deepest-path
                     acceptance (Sec. 2.4 greedy rule; App. E).
  draft_topw,     -- budgeted tree drafting: top-W candidates per draft depth
  build_tree         and best-first expansion by accumulated draft
                     log-probability (Sec. 2.4 parallel tree drafting; Alg. 1).
  kv_commit       -- the cache side: committing the accepted path, paged
                     caches, the tree-tail layout (App. E).
  tree_accept_sampled -- non-greedy (temperature) tree acceptance: the
                     speculative sampling rule (Sec. 2.4) applied to each
                     node's deterministic children in turn against the
                     target's residual, which keeps verification lossless
                     (Sec. 2.2); correction token drawn from the final
                     residual; philox -- its counter-based random numbers
                     (Salmon et al. 2011).
  block_causal    -- attention under the draft head's training mask: anchor
                     blocks that see the prefix before their anchor and
                     their own earlier positions (App. Training Details).
  brute           -- pure-Python loop versions for tiny inputs, used only to
                     pin the functions above.

Parity is pinned for every function (brute force, closed forms, invariants
and library special cases in the tests).
"""
from .tree_attention import (decode_bf16, tree_structure, full_mask,
                             tree_attention)
from .tree_accept import target_argmax, tree_accept
from .tree_build import draft_topw, build_tree
from .tree_accept_sampled import tree_accept_sampled
from .block_causal import training_mask, block_causal_attention
from .kv_commit import commit_path, gather_paged, commit_path_paged, tree_tail, commit_path_tail

__all__ = ["decode_bf16", "tree_structure", "full_mask", "tree_attention",
           "target_argmax", "tree_accept", "draft_topw", "build_tree",
           "commit_path", "gather_paged", "commit_path_paged", "tree_tail",
           "commit_path_tail", "training_mask", "block_causal_attention",
           "tree_accept_sampled"]
