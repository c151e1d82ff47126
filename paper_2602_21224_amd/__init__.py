"""Target-model tree verification for MI355X (gfx950): HIP kernels behind a C ABI.

The entry points are re-exported lazily from `_lib` so that importing the
package (for example to draw synthetic workloads) does not need the built
library.
"""

__all__ = ["tree_verify_attention", "tree_argmax_accept", "tree_argmax_accept_noalloc",
           "kv_compact_accepted",
           "tv_validate_inputs", "tree_build", "tree_resample", "tree_lm_head_argmax_accept",
           "attention_workspace_size", "lm_head_workspace_size",
           "argmax_workspace_size", "tree_build_workspace_size", "abi_version", "load"]


def __getattr__(name):
    if name in __all__:
        from . import _lib
        return getattr(_lib, name)
    raise AttributeError(name)
