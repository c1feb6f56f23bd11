"""ctypes binding of libtv (include/tv.h). Argument marshalling only."""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtv.so")

TV_OK, TV_ERR_INVALID_ARG, TV_ERR_UNSUPPORTED, TV_ERR_WORKSPACE, TV_ERR_HIP = range(5)
TV_DTYPE_BF16, TV_DTYPE_F32 = 0, 1
TV_SIBLINGS_WITHOUT_REPLACEMENT, TV_SIBLINGS_WITH_REPLACEMENT = 0, 1
(TV_TREE_OK, TV_TREE_BAD_PARENT, TV_TREE_BAD_TOKEN, TV_TREE_DUP_SIBLING, TV_TREE_NONFINITE,
 TV_TREE_DEGENERATE, TV_TREE_ABORTED) = range(7)
TV_NODE_UNTESTED, TV_NODE_ACCEPTED, TV_NODE_REJECTED, TV_NODE_PRUNED = range(4)
TV_MAX_BATCH = 1 << 20
TV_MAX_NODES = 1024
TV_MAX_VOCAB = 1 << 20
TV_MAX_VOCAB_F32 = 1 << 19
TV_NUM_COUNTERS = 4
TV_MAX_LMHEAD_ROWS = 1 << 18
TV_MAX_HIDDEN = 1 << 16


class TvError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {tv_status_string(code)} (status {code})")
        self.code = code


_lib = None

_VERIFY_ARGTYPES = [
    ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,            # batch, num_nodes, vocab
    ctypes.c_void_p, ctypes.c_void_p,                          # parents, tokens
    ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,          # target, draft, dtype
    ctypes.c_float, ctypes.c_void_p, ctypes.c_int32,           # temperature, uniforms, mode
    ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,         # accept_len, node, bonus
    ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,         # status, node_state, theta
    ctypes.c_void_p, ctypes.c_void_p,                          # p_init, counters
    ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,         # workspace, bytes, stream
]


_SAMPLE_ARGTYPES = [
    ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,            # batch, num_nodes, vocab
    ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,          # parents, draft, dtype
    ctypes.c_float, ctypes.c_void_p, ctypes.c_int32,           # temperature, uniforms, mode
    ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,         # tokens, status, stream
]


def load_library(path: str = LIB_PATH):
    """Load libtv.so once. Raises if it is not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing; build it with __graft_entry__.build()")
        lib = ctypes.CDLL(path)
        lib.tv_workspace_size.argtypes = [ctypes.c_int32] * 3
        lib.tv_workspace_size.restype = ctypes.c_size_t
        for name in ("tv_verify", "tv_verify_tokenlevel"):
            fn = getattr(lib, name)
            fn.argtypes = _VERIFY_ARGTYPES
            fn.restype = ctypes.c_int
        lib.tv_verify_noalloc.argtypes = _VERIFY_ARGTYPES[:19] + [ctypes.c_void_p]
        lib.tv_verify_noalloc.restype = ctypes.c_int
        lib.tv_verify_stats.argtypes = (_VERIFY_ARGTYPES[:11] + [ctypes.c_void_p] * 4 +
                                        _VERIFY_ARGTYPES[11:])
        lib.tv_verify_stats.restype = ctypes.c_int
        lib.tv_lmhead_workspace_size.argtypes = [ctypes.c_int32, ctypes.c_int32]
        lib.tv_lmhead_workspace_size.restype = ctypes.c_size_t
        lib.tv_lmhead_stats.argtypes = [ctypes.c_int32] * 3 + [ctypes.c_void_p] * 2 + \
            [ctypes.c_float] + [ctypes.c_void_p] * 4 + [ctypes.c_size_t, ctypes.c_void_p]
        lib.tv_lmhead_stats.restype = ctypes.c_int
        lib.tv_draft_tokens.argtypes = _SAMPLE_ARGTYPES
        lib.tv_draft_tokens.restype = ctypes.c_int
        lib.tv_commit_paths.argtypes = [ctypes.c_int32, ctypes.c_int32] + \
            [ctypes.c_void_p] * 5 + [ctypes.c_int32] + [ctypes.c_void_p] * 4
        lib.tv_commit_paths.restype = ctypes.c_int
        lib.tv_status_string.argtypes = [ctypes.c_int]
        lib.tv_status_string.restype = ctypes.c_char_p
        _lib = lib
    return _lib


def tv_status_string(code: int) -> str:
    return load_library().tv_status_string(int(code)).decode()


def tv_workspace_size(batch: int, num_nodes: int, vocab: int) -> int:
    return int(load_library().tv_workspace_size(batch, num_nodes, vocab))


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _dtype_code(t):
    import torch
    if t.dtype == torch.bfloat16:
        return TV_DTYPE_BF16
    if t.dtype == torch.float32:
        return TV_DTYPE_F32
    raise TypeError(f"logits must be bfloat16 or float32, got {t.dtype}")


def _call(name, batch, num_nodes, vocab, parents, tokens, target_logits, draft_logits, dtype,
          temperature, uniforms, mode, accept_len, accepted_node, bonus_token, status,
          node_state, node_theta, p_init, counters, workspace, workspace_bytes, stream):
    fn = getattr(load_library(), name)
    return int(fn(batch, num_nodes, vocab, _ptr(parents), _ptr(tokens), _ptr(target_logits),
                  _ptr(draft_logits), dtype, float(temperature), _ptr(uniforms), mode,
                  _ptr(accept_len), _ptr(accepted_node), _ptr(bonus_token), _ptr(status),
                  _ptr(node_state), _ptr(node_theta), _ptr(p_init), _ptr(counters),
                  _ptr(workspace), int(workspace_bytes), stream))


def tv_verify(batch, num_nodes, vocab, parents, tokens, target_logits, draft_logits, dtype,
              temperature, uniforms, mode, accept_len, accepted_node, bonus_token, status,
              node_state=None, node_theta=None, p_init=None, counters=None, workspace=None,
              workspace_bytes=0, stream=None) -> int:
    """C-ABI ``tv_verify``: pointers may be torch tensors or raw ints; returns the status."""
    return _call("tv_verify", batch, num_nodes, vocab, parents, tokens, target_logits,
                 draft_logits, dtype, temperature, uniforms, mode, accept_len, accepted_node,
                 bonus_token, status, node_state, node_theta, p_init, counters, workspace,
                 workspace_bytes, stream)


def tv_verify_noalloc(batch, num_nodes, vocab, parents, tokens, target_logits, draft_logits,
                      dtype, temperature, uniforms, mode, accept_len, accepted_node, bonus_token,
                      status, node_state=None, node_theta=None, p_init=None, counters=None,
                      stream=None) -> int:
    """C-ABI ``tv_verify_noalloc``: ``tv_verify`` on the library's own device
    scratch (no workspace argument); returns the status."""
    fn = load_library().tv_verify_noalloc
    return int(fn(batch, num_nodes, vocab, _ptr(parents), _ptr(tokens), _ptr(target_logits),
                  _ptr(draft_logits), dtype, float(temperature), _ptr(uniforms), mode,
                  _ptr(accept_len), _ptr(accepted_node), _ptr(bonus_token), _ptr(status),
                  _ptr(node_state), _ptr(node_theta), _ptr(p_init), _ptr(counters), stream))


def tv_verify_stats(batch, num_nodes, vocab, parents, tokens, target_logits, draft_logits,
                    dtype, temperature, uniforms, mode, target_max, target_sum, draft_max,
                    draft_sum, accept_len, accepted_node, bonus_token, status, node_state=None,
                    node_theta=None, p_init=None, counters=None, workspace=None,
                    workspace_bytes=0, stream=None) -> int:
    """C-ABI ``tv_verify_stats``: ``tv_verify`` with the row statistics given."""
    fn = load_library().tv_verify_stats
    return int(fn(batch, num_nodes, vocab, _ptr(parents), _ptr(tokens), _ptr(target_logits),
                  _ptr(draft_logits), dtype, float(temperature), _ptr(uniforms), mode,
                  _ptr(target_max), _ptr(target_sum), _ptr(draft_max), _ptr(draft_sum),
                  _ptr(accept_len), _ptr(accepted_node), _ptr(bonus_token), _ptr(status),
                  _ptr(node_state), _ptr(node_theta), _ptr(p_init), _ptr(counters),
                  _ptr(workspace), int(workspace_bytes), stream))


def tv_lmhead_workspace_size(rows: int, vocab: int) -> int:
    return int(load_library().tv_lmhead_workspace_size(rows, vocab))


def tv_lmhead_stats(rows, hidden_size, vocab, hidden, weight, temperature, logits, row_max,
                    row_sum, workspace, workspace_bytes, stream=None) -> int:
    """C-ABI ``tv_lmhead_stats``: pointers may be torch tensors or raw ints."""
    return int(load_library().tv_lmhead_stats(
        int(rows), int(hidden_size), int(vocab), _ptr(hidden), _ptr(weight), float(temperature),
        _ptr(logits), _ptr(row_max), _ptr(row_sum), _ptr(workspace), int(workspace_bytes),
        _ptr(stream)))


def lmhead_stats(hidden, weight, temperature, stream=None, out=None):
    """Logits and their row statistics for bf16 hidden states [..., K] and a bf16
    weight [N, K] (torch tensors on one device); returns (logits [..., N] bf16,
    row_max [...] float32, row_sum [...] float64). Raises on a non-OK return."""
    import torch
    K = hidden.shape[-1]
    N = weight.shape[0]
    lead = tuple(hidden.shape[:-1])
    M = 1
    for d in lead:
        M *= d
    dev = hidden.device
    if hidden.dtype != torch.bfloat16 or weight.dtype != torch.bfloat16:
        raise TypeError("hidden and weight must be bfloat16")
    if tuple(weight.shape) != (N, K) or not hidden.is_contiguous() or not weight.is_contiguous():
        raise ValueError("weight must be [vocab, hidden] and both tensors contiguous")
    if out is None:
        out = (torch.empty(lead + (N,), dtype=torch.bfloat16, device=dev),
               torch.empty(lead, dtype=torch.float32, device=dev),
               torch.empty(lead, dtype=torch.float64, device=dev))
    nbytes = tv_lmhead_workspace_size(M, N)
    ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    if stream is None:
        stream = torch.cuda.current_stream(dev).cuda_stream if dev.type == "cuda" else None
    st = tv_lmhead_stats(M, K, N, hidden, weight, temperature, out[0], out[1], out[2], ws, nbytes,
                         stream)
    if st != TV_OK:
        raise TvError(st, "tv_lmhead_stats")
    return out


def tv_verify_tokenlevel(batch, num_nodes, vocab, parents, tokens, target_logits, draft_logits,
                         dtype, temperature, uniforms, mode, accept_len, accepted_node,
                         bonus_token, status, node_state=None, node_theta=None, p_init=None,
                         counters=None, workspace=None, workspace_bytes=0, stream=None) -> int:
    """C-ABI ``tv_verify_tokenlevel``; same arguments as :func:`tv_verify`."""
    return _call("tv_verify_tokenlevel", batch, num_nodes, vocab, parents, tokens,
                 target_logits, draft_logits, dtype, temperature, uniforms, mode, accept_len,
                 accepted_node, bonus_token, status, node_state, node_theta, p_init, counters,
                 workspace, workspace_bytes, stream)


def tv_draft_tokens(batch, num_nodes, vocab, parents, draft_logits, dtype, temperature,
                    uniforms, mode, tokens, status, stream=None) -> int:
    """C-ABI ``tv_draft_tokens``: pointers may be torch tensors or raw ints;
    returns the status."""
    return int(load_library().tv_draft_tokens(
        int(batch), int(num_nodes), int(vocab), _ptr(parents), _ptr(draft_logits), int(dtype),
        float(temperature), _ptr(uniforms), int(mode), _ptr(tokens), _ptr(status),
        _ptr(stream)))


def draft_tokens(parents, draft_logits, temperature, uniforms, mode, stream=None):
    """Draws the tokens of a batch of draft trees on the device (torch tensors
    in, (tokens, status) int32 tensors out); raises on a non-OK return."""
    import torch
    B, n1 = parents.shape
    V = draft_logits.shape[-1]
    dev = draft_logits.device
    for name, t, shape in (("parents", parents, (B, n1)), ("uniforms", uniforms, (B, n1)),
                           ("draft_logits", draft_logits, (B, n1, V))):
        if tuple(t.shape) != shape:
            raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {shape}")
        if t.device != dev or not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous on {dev}")
    if parents.dtype != torch.int32 or uniforms.dtype != torch.float32:
        raise TypeError("parents must be int32 and uniforms float32")
    tokens = torch.empty((B, n1), dtype=torch.int32, device=dev)
    status = torch.empty(B, dtype=torch.int32, device=dev)
    if stream is None:
        stream = torch.cuda.current_stream(dev).cuda_stream if dev.type == "cuda" else None
    st = tv_draft_tokens(B, n1, V, parents, draft_logits, _dtype_code(draft_logits), temperature,
                         uniforms, mode, tokens, status, stream)
    if st != TV_OK:
        raise TvError(st, "tv_draft_tokens")
    return tokens, status


TV_COMMIT_OVERFLOW, TV_COMMIT_INCONSISTENT = -1, -2


def tv_commit_paths(batch, num_nodes, parents, tokens, accepted_node, bonus_token, status,
                    max_len, path_nodes, path_tokens, path_len, stream=None) -> int:
    """C-ABI ``tv_commit_paths``: pointers may be torch tensors or raw ints;
    returns the status."""
    return int(load_library().tv_commit_paths(
        int(batch), int(num_nodes), _ptr(parents), _ptr(tokens), _ptr(accepted_node),
        _ptr(bonus_token), _ptr(status), int(max_len), _ptr(path_nodes), _ptr(path_tokens),
        _ptr(path_len), _ptr(stream)))


def commit_paths(parents, tokens, out: "VerifyOutputs", max_len: int, stream=None):
    """The committed chain of every tree after a verification (torch tensors
    in; (path_nodes, path_tokens, path_len) int32 tensors out); raises on a
    non-OK return."""
    import torch
    B, n1 = parents.shape
    dev = parents.device
    pn = torch.empty((B, max(max_len, 1)), dtype=torch.int32, device=dev)
    pt = torch.empty((B, max_len + 1), dtype=torch.int32, device=dev)
    pl = torch.empty(B, dtype=torch.int32, device=dev)
    if stream is None:
        stream = torch.cuda.current_stream(dev).cuda_stream if dev.type == "cuda" else None
    st = tv_commit_paths(B, n1, parents, tokens, out.accepted_node, out.bonus_token, out.status,
                         max_len, pn, pt, pl, stream)
    if st != TV_OK:
        raise TvError(st, "tv_commit_paths")
    return pn[:, :max_len], pt, pl


def workspace_tensor(batch: int, num_nodes: int, vocab: int, device):
    """A device buffer of tv_workspace_size() bytes (torch allocations are
    256-byte aligned)."""
    import torch
    n = tv_workspace_size(batch, num_nodes, vocab)
    return torch.empty(max(n, 1), dtype=torch.uint8, device=device), n


@dataclass
class VerifyOutputs:
    accept_len: object
    accepted_node: object
    bonus_token: object
    status: object
    node_state: object = None
    node_theta: object = None
    p_init: object = None
    counters: object = None


def verify_batch(parents, tokens, target_logits, draft_logits, temperature, uniforms, mode,
                 tokenlevel=False, want_nodes=True, want_p_init=False, want_counters=True,
                 out: VerifyOutputs | None = None, stream=None,
                 workspace=None, want_theta=None, stats=None) -> VerifyOutputs:
    """Allocate outputs and the workspace (torch, same device) unless given,
    check shapes, call the C entry point on the current stream and raise on a
    non-OK return. ``want_nodes`` asks for node states and (unless
    ``want_theta`` is False) the tested probabilities; without the latter,
    tv_verify skips the residual updates that decide nothing. ``stats`` =
    (target_max, target_sum, draft_max, draft_sum) [B, N+1] tensors calls
    tv_verify_stats (Traversal Verification with the row statistics given)."""
    import torch
    B, n1 = parents.shape
    V = target_logits.shape[-1]
    dev = target_logits.device
    for name, t, shape in (("parents", parents, (B, n1)), ("tokens", tokens, (B, n1)),
                           ("uniforms", uniforms, (B, n1)),
                           ("target_logits", target_logits, (B, n1, V)),
                           ("draft_logits", draft_logits, (B, n1, V))):
        if tuple(t.shape) != shape:
            raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {shape}")
        if t.device != dev or not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous on {dev}")
    if parents.dtype != torch.int32 or tokens.dtype != torch.int32:
        raise TypeError("parents and tokens must be int32")
    if uniforms.dtype != torch.float32:
        raise TypeError("uniforms must be float32")
    if draft_logits.dtype != target_logits.dtype:
        raise TypeError("target and draft logits must share a dtype")
    dtype = _dtype_code(target_logits)
    if out is None:
        i32 = dict(dtype=torch.int32, device=dev)
        out = VerifyOutputs(
            accept_len=torch.empty(B, **i32), accepted_node=torch.empty(B, **i32),
            bonus_token=torch.empty(B, **i32), status=torch.empty(B, **i32),
            node_state=torch.empty((B, n1), dtype=torch.int8, device=dev) if want_nodes else None,
            node_theta=torch.empty((B, n1), dtype=torch.float32, device=dev)
            if (want_nodes if want_theta is None else want_theta) else None,
            p_init=torch.empty((B, n1), dtype=torch.float32, device=dev) if want_p_init else None,
            counters=torch.empty((B, TV_NUM_COUNTERS), **i32) if want_counters else None)
    if stream is None:
        stream = torch.cuda.current_stream(dev).cuda_stream if dev.type == "cuda" else None
    if workspace is None:
        workspace, ws_bytes = workspace_tensor(B, n1, V, dev)
    else:
        ws_bytes = workspace.numel() * workspace.element_size()
    if stats is not None:
        if tokenlevel:
            raise ValueError("row statistics are taken by Traversal Verification only")
        tm, ts, dm, ds = stats
        for name, t, dt in (("target_max", tm, torch.float32), ("target_sum", ts, torch.float64),
                            ("draft_max", dm, torch.float32), ("draft_sum", ds, torch.float64)):
            if tuple(t.shape) != (B, n1) or t.dtype != dt or not t.is_contiguous():
                raise ValueError(f"{name} must be a contiguous {dt} tensor of shape {(B, n1)}")
        st = tv_verify_stats(B, n1, V, parents, tokens, target_logits, draft_logits, dtype,
                             temperature, uniforms, mode, tm, ts, dm, ds, out.accept_len,
                             out.accepted_node, out.bonus_token, out.status, out.node_state,
                             out.node_theta, out.p_init, out.counters, workspace, ws_bytes,
                             stream)
        if st != TV_OK:
            raise TvError(st, "tv_verify_stats")
        return out
    fn = tv_verify_tokenlevel if tokenlevel else tv_verify
    st = fn(B, n1, V, parents, tokens, target_logits, draft_logits, dtype, temperature,
            uniforms, mode, out.accept_len, out.accepted_node, out.bonus_token, out.status,
            out.node_state, out.node_theta, out.p_init, out.counters, workspace, ws_bytes,
            stream)
    if st != TV_OK:
        raise TvError(st, fn.__name__)
    return out
