"""MI355X-native tree verification for parallel tree drafting speculative
decoding: tree-masked GQA attention and greedy tree acceptance as HIP kernels
for gfx950 behind a C ABI (include/treeverify.h).

Importing the package loads nothing; the first call loads libtreeverify.so
and raises if it is missing.
"""

__all__ = ["tree_verify_attention", "tree_verify_attention_paged", "tree_accept",
           "commit_path", "commit_path_paged", "draft_topw", "build_tree",
           "block_causal_attention", "tree_accept_sampled", "load_library"]


def tree_verify_attention(*args, **kwargs):
    from .binding import tree_verify_attention as f
    return f(*args, **kwargs)


def tree_verify_attention_paged(*args, **kwargs):
    from .binding import tree_verify_attention_paged as f
    return f(*args, **kwargs)


def commit_path(*args, **kwargs):
    from .binding import commit_path as f
    return f(*args, **kwargs)


def commit_path_paged(*args, **kwargs):
    from .binding import commit_path_paged as f
    return f(*args, **kwargs)


def tree_accept(*args, **kwargs):
    from .binding import tree_accept as f
    return f(*args, **kwargs)


def draft_topw(*args, **kwargs):
    from .binding import draft_topw as f
    return f(*args, **kwargs)


def build_tree(*args, **kwargs):
    from .binding import build_tree as f
    return f(*args, **kwargs)


def block_causal_attention(*args, **kwargs):
    from .binding import block_causal_attention as f
    return f(*args, **kwargs)


def tree_accept_sampled(*args, **kwargs):
    from .binding import tree_accept_sampled as f
    return f(*args, **kwargs)


def load_library():
    from .binding import load_library as f
    return f()
