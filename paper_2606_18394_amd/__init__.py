"""MI355X-native tree verification for parallel tree drafting speculative
decoding: tree-masked GQA attention and greedy tree acceptance as HIP kernels
for gfx950 behind a C ABI (include/treeverify.h).

Importing the package loads nothing; the first call loads libtreeverify.so
and raises if it is missing.  The public calls are those of ``binding``.
"""

__all__ = ["tree_verify_attention", "tree_verify_attention_paged", "tree_accept",
           "tree_accept_noalloc", "commit_path", "commit_path_paged", "draft_topw",
           "build_tree", "block_causal_attention", "tree_accept_sampled", "load_library"]


def __getattr__(name):
    # lazy: torch and the library load on first use of a call
    if name in __all__:
        from . import binding
        return getattr(binding, name)
    raise AttributeError(f"module {__name__!r} has no attribute {name!r}")
