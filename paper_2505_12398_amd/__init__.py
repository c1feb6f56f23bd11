"""Batched Traversal Verification (arXiv 2505.12398) on MI355X.

The work happens in ``libtv.so`` (HIP kernels for gfx950 behind the C-ABI in
``include/tv.h``). This package is a thin ctypes binding with the same names
as the C entry points; torch tensors supply device memory and the stream.
There is no fallback: if the library is missing or fails to load, every call
raises.
"""

from ._lib import (  # noqa: F401
    TV_OK, TV_ERR_INVALID_ARG, TV_ERR_UNSUPPORTED, TV_ERR_WORKSPACE, TV_ERR_HIP,
    TV_DTYPE_BF16, TV_DTYPE_F32,
    TV_SIBLINGS_WITHOUT_REPLACEMENT, TV_SIBLINGS_WITH_REPLACEMENT,
    TV_TREE_OK, TV_TREE_BAD_PARENT, TV_TREE_BAD_TOKEN, TV_TREE_DUP_SIBLING,
    TV_TREE_NONFINITE, TV_TREE_DEGENERATE, TV_TREE_ABORTED,
    TV_NODE_UNTESTED, TV_NODE_ACCEPTED, TV_NODE_REJECTED, TV_NODE_PRUNED,
    TV_MAX_BATCH, TV_MAX_NODES, TV_MAX_VOCAB, TV_MAX_VOCAB_F32, TV_NUM_COUNTERS,
    LIB_PATH, TvError, load_library,
    tv_workspace_size, tv_verify, tv_verify_noalloc, tv_verify_tokenlevel, tv_status_string, tv_draft_tokens,
    draft_tokens, tv_commit_paths, commit_paths, TV_COMMIT_OVERFLOW, TV_COMMIT_INCONSISTENT,
    VerifyOutputs, verify_batch, workspace_tensor, tv_verify_stats, tv_lmhead_workspace_size,
    tv_lmhead_stats, lmhead_stats, TV_MAX_LMHEAD_ROWS, TV_MAX_HIDDEN,
)
