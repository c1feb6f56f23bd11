"""The C-ABI library without a GPU: it loads, exports every function the
header declares, agrees with the binding's constants, and rejects bad
arguments on the host before any HIP call."""

import ctypes
import os
import re

import pytest

import paper_2505_12398_amd as tv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tv.h")


def header_text():
    with open(HEADER) as f:
        return f.read()


def declared_functions():
    text = re.sub(r"/\*.*?\*/", "", header_text(), flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:size_t|int|const char\*)\s+(tv_\w+)\s*\(", text,
                                 flags=re.M)))


def test_library_exports_every_declared_function():
    lib = tv.load_library()
    names = declared_functions()
    assert {"tv_verify", "tv_verify_tokenlevel", "tv_workspace_size",
            "tv_status_string", "tv_draft_tokens"} <= set(names)
    for name in names:
        assert hasattr(lib, name), name


def test_constants_match_header():
    text = header_text()

    def define(name):
        line = re.search(rf"#define {name}\s+([^\n]+)", text).group(1)
        return line.split("/*")[0].strip()

    assert eval(define("TV_MAX_BATCH")) == tv.TV_MAX_BATCH
    assert eval(define("TV_MAX_NODES")) == tv.TV_MAX_NODES
    assert eval(define("TV_MAX_VOCAB")) == tv.TV_MAX_VOCAB
    assert eval(define("TV_MAX_VOCAB_F32")) == tv.TV_MAX_VOCAB_F32
    assert eval(define("TV_NUM_COUNTERS")) == tv.TV_NUM_COUNTERS
    for name in ["TV_OK", "TV_ERR_INVALID_ARG", "TV_ERR_UNSUPPORTED", "TV_ERR_WORKSPACE",
                 "TV_ERR_HIP", "TV_DTYPE_BF16", "TV_DTYPE_F32", "TV_SIBLINGS_WITHOUT_REPLACEMENT",
                 "TV_SIBLINGS_WITH_REPLACEMENT", "TV_TREE_OK", "TV_TREE_BAD_PARENT",
                 "TV_TREE_BAD_TOKEN", "TV_TREE_DUP_SIBLING", "TV_TREE_NONFINITE",
                 "TV_TREE_DEGENERATE", "TV_TREE_ABORTED", "TV_NODE_UNTESTED", "TV_NODE_ACCEPTED",
                 "TV_NODE_REJECTED", "TV_NODE_PRUNED"]:
        m = re.search(rf"\b{name}\s*=\s*(\d+)", text)
        assert m and int(m.group(1)) == getattr(tv, name), name


def test_status_strings():
    assert tv.tv_status_string(tv.TV_OK) == "ok"
    for code in range(1, 5):
        assert tv.tv_status_string(code) not in ("ok", "unknown status")
    assert tv.tv_status_string(99) == "unknown status"


def test_workspace_size():
    ws = tv.tv_workspace_size
    # invalid sizes report 0
    for args in [(0, 65, 1000), (-1, 65, 1000), (1, 0, 1000), (1, tv.TV_MAX_NODES + 1, 1000),
                 (1, 65, 1), (1, 65, tv.TV_MAX_VOCAB + 1), (tv.TV_MAX_BATCH + 1, 65, 1000)]:
        assert ws(*args) == 0, args
    # positive, 256-byte granular, monotone in batch and vocabulary, bounded
    sizes = [ws(b, 65, 128256) for b in (1, 2, 16, 256, 4096, tv.TV_MAX_BATCH)]
    assert all(s > 0 and s % 256 == 0 for s in sizes)
    assert sizes == sorted(sizes)
    assert sizes[-1] == sizes[-2]          # capped by the number of workgroups per call
    assert ws(16, 65, 2) <= ws(16, 65, 128256) <= ws(16, 65, tv.TV_MAX_VOCAB)
    assert ws(tv.TV_MAX_BATCH, tv.TV_MAX_NODES, tv.TV_MAX_VOCAB) <= 3 << 20
    # independent of the tree size
    assert ws(256, 2, 128256) == ws(256, tv.TV_MAX_NODES, 128256)


# Fake, never-dereferenced device addresses: validation fails before any HIP call.
A = 0x10000
WS = 0x40000000


def call(fn="tv_verify", **kw):
    args = dict(batch=2, num_nodes=5, vocab=100, parents=A, tokens=A, target_logits=A,
                draft_logits=A + 0x1000, dtype=tv.TV_DTYPE_BF16, temperature=1.0, uniforms=A,
                mode=0, accept_len=A, accepted_node=A, bonus_token=A, status=A,
                workspace=WS, workspace_bytes=tv.tv_workspace_size(2, 5, 100))
    args.update(kw)
    return getattr(tv, fn)(**args)


@pytest.mark.parametrize("fn", ["tv_verify", "tv_verify_tokenlevel"])
@pytest.mark.parametrize("kw,want", [
    (dict(batch=-1), tv.TV_ERR_INVALID_ARG),
    (dict(num_nodes=0), tv.TV_ERR_INVALID_ARG),
    (dict(vocab=1), tv.TV_ERR_INVALID_ARG),
    (dict(dtype=7), tv.TV_ERR_INVALID_ARG),
    (dict(mode=2), tv.TV_ERR_INVALID_ARG),
    (dict(temperature=0.0), tv.TV_ERR_INVALID_ARG),
    (dict(temperature=-1.0), tv.TV_ERR_INVALID_ARG),
    (dict(temperature=float("nan")), tv.TV_ERR_INVALID_ARG),
    (dict(temperature=float("inf")), tv.TV_ERR_INVALID_ARG),
    (dict(temperature=1e-5), tv.TV_ERR_UNSUPPORTED),
    (dict(temperature=1e4), tv.TV_ERR_UNSUPPORTED),
    (dict(num_nodes=tv.TV_MAX_NODES + 1), tv.TV_ERR_UNSUPPORTED),
    (dict(vocab=tv.TV_MAX_VOCAB + 1), tv.TV_ERR_UNSUPPORTED),
    (dict(dtype=tv.TV_DTYPE_F32, vocab=tv.TV_MAX_VOCAB_F32 + 1), tv.TV_ERR_UNSUPPORTED),
    (dict(parents=None), tv.TV_ERR_INVALID_ARG),
    (dict(tokens=None), tv.TV_ERR_INVALID_ARG),
    (dict(target_logits=None), tv.TV_ERR_INVALID_ARG),
    (dict(draft_logits=None), tv.TV_ERR_INVALID_ARG),
    (dict(uniforms=None), tv.TV_ERR_INVALID_ARG),
    (dict(accept_len=None), tv.TV_ERR_INVALID_ARG),
    (dict(accepted_node=None), tv.TV_ERR_INVALID_ARG),
    (dict(bonus_token=None), tv.TV_ERR_INVALID_ARG),
    (dict(status=None), tv.TV_ERR_INVALID_ARG),
    (dict(target_logits=A + 1, draft_logits=A + 1), tv.TV_ERR_INVALID_ARG),
    (dict(dtype=tv.TV_DTYPE_F32, target_logits=A + 2, draft_logits=A + 2),
     tv.TV_ERR_INVALID_ARG),
    (dict(target_logits=A + 2, draft_logits=A + 4), tv.TV_ERR_UNSUPPORTED),
    (dict(parents=A + 2), tv.TV_ERR_INVALID_ARG),
    (dict(counters=A + 1), tv.TV_ERR_INVALID_ARG),
    (dict(batch=tv.TV_MAX_BATCH + 1), tv.TV_ERR_UNSUPPORTED),
    (dict(workspace=None), tv.TV_ERR_WORKSPACE),
    (dict(workspace=WS + 128), tv.TV_ERR_WORKSPACE),
    (dict(workspace_bytes=256), tv.TV_ERR_WORKSPACE),
])
def test_host_validation(fn, kw, want):
    assert call(fn, **kw) == want


@pytest.mark.parametrize("fn", ["tv_verify", "tv_verify_tokenlevel"])
def test_empty_batch_is_a_no_op(fn):
    # batch 0 with null buffers: valid, nothing enqueued, no HIP call
    assert call(fn, batch=0, parents=None, tokens=None, target_logits=None, draft_logits=None,
                uniforms=None, accept_len=None, accepted_node=None, bonus_token=None,
                status=None) == tv.TV_OK


def call_sampler(**kw):
    args = dict(batch=2, num_nodes=5, vocab=100, parents=A, draft_logits=A + 0x1000,
                dtype=tv.TV_DTYPE_BF16, temperature=1.0, uniforms=A, mode=0, tokens=A, status=A)
    args.update(kw)
    return tv.tv_draft_tokens(**args)


@pytest.mark.parametrize("kw,want", [
    (dict(batch=-1), tv.TV_ERR_INVALID_ARG),
    (dict(num_nodes=0), tv.TV_ERR_INVALID_ARG),
    (dict(vocab=1), tv.TV_ERR_INVALID_ARG),
    (dict(dtype=7), tv.TV_ERR_INVALID_ARG),
    (dict(mode=2), tv.TV_ERR_INVALID_ARG),
    (dict(temperature=0.0), tv.TV_ERR_INVALID_ARG),
    (dict(temperature=float("nan")), tv.TV_ERR_INVALID_ARG),
    (dict(temperature=1e-5), tv.TV_ERR_UNSUPPORTED),
    (dict(num_nodes=tv.TV_MAX_NODES + 1), tv.TV_ERR_UNSUPPORTED),
    (dict(vocab=tv.TV_MAX_VOCAB + 1), tv.TV_ERR_UNSUPPORTED),
    (dict(batch=tv.TV_MAX_BATCH + 1), tv.TV_ERR_UNSUPPORTED),
    (dict(parents=None), tv.TV_ERR_INVALID_ARG),
    (dict(draft_logits=None), tv.TV_ERR_INVALID_ARG),
    (dict(uniforms=None), tv.TV_ERR_INVALID_ARG),
    (dict(tokens=None), tv.TV_ERR_INVALID_ARG),
    (dict(status=None), tv.TV_ERR_INVALID_ARG),
    (dict(draft_logits=A + 1), tv.TV_ERR_INVALID_ARG),
    (dict(tokens=A + 2), tv.TV_ERR_INVALID_ARG),
])
def test_sampler_argument_errors_launch_nothing(kw, want):
    """Host-side validation of tv_draft_tokens returns before any HIP call (no GPU here)."""
    assert call_sampler(**kw) == want


def test_sampler_empty_batch_is_ok():
    assert call_sampler(batch=0, parents=None, draft_logits=None, uniforms=None, tokens=None,
                        status=None) == tv.TV_OK


def call_commit(**kw):
    args = dict(batch=2, num_nodes=5, parents=A, tokens=A, accepted_node=A, bonus_token=A,
                status=A, max_len=4, path_nodes=A, path_tokens=A, path_len=A)
    args.update(kw)
    return tv.tv_commit_paths(**args)


@pytest.mark.parametrize("kw,want", [
    (dict(batch=-1), tv.TV_ERR_INVALID_ARG),
    (dict(num_nodes=0), tv.TV_ERR_INVALID_ARG),
    (dict(max_len=-1), tv.TV_ERR_INVALID_ARG),
    (dict(num_nodes=tv.TV_MAX_NODES + 1), tv.TV_ERR_UNSUPPORTED),
    (dict(max_len=tv.TV_MAX_NODES + 1), tv.TV_ERR_UNSUPPORTED),
    (dict(parents=None), tv.TV_ERR_INVALID_ARG),
    (dict(accepted_node=None), tv.TV_ERR_INVALID_ARG),
    (dict(path_tokens=None), tv.TV_ERR_INVALID_ARG),
    (dict(path_nodes=None), tv.TV_ERR_INVALID_ARG),
    (dict(path_len=A + 2), tv.TV_ERR_INVALID_ARG),
])
def test_commit_argument_errors_launch_nothing(kw, want):
    """Host-side validation of tv_commit_paths returns before any HIP call (no GPU here)."""
    assert call_commit(**kw) == want


def test_commit_empty_batch_is_ok():
    assert call_commit(batch=0, parents=None, tokens=None) == tv.TV_OK


def call_noalloc(**kw):
    args = dict(batch=2, num_nodes=5, vocab=100, parents=A, tokens=A, target_logits=A,
                draft_logits=A + 0x1000, dtype=tv.TV_DTYPE_BF16, temperature=1.0, uniforms=A,
                mode=0, accept_len=A, accepted_node=A, bonus_token=A, status=A)
    args.update(kw)
    return tv.tv_verify_noalloc(**args)


@pytest.mark.parametrize("kw,want", [
    (dict(batch=-1), tv.TV_ERR_INVALID_ARG),
    (dict(num_nodes=0), tv.TV_ERR_INVALID_ARG),
    (dict(vocab=1), tv.TV_ERR_INVALID_ARG),
    (dict(dtype=7), tv.TV_ERR_INVALID_ARG),
    (dict(mode=2), tv.TV_ERR_INVALID_ARG),
    (dict(temperature=float("nan")), tv.TV_ERR_INVALID_ARG),
    (dict(temperature=1e-5), tv.TV_ERR_UNSUPPORTED),
    (dict(num_nodes=tv.TV_MAX_NODES + 1), tv.TV_ERR_UNSUPPORTED),
    (dict(batch=tv.TV_MAX_BATCH + 1), tv.TV_ERR_UNSUPPORTED),
    (dict(parents=None), tv.TV_ERR_INVALID_ARG),
    (dict(status=None), tv.TV_ERR_INVALID_ARG),
    (dict(target_logits=A + 2, draft_logits=A + 4), tv.TV_ERR_UNSUPPORTED),
    (dict(counters=A + 1), tv.TV_ERR_INVALID_ARG),
])
def test_noalloc_argument_errors_launch_nothing(kw, want):
    """tv_verify_noalloc checks its arguments on the host before it looks up
    its device scratch (no GPU here)."""
    assert call_noalloc(**kw) == want


def test_noalloc_empty_batch_is_ok():
    assert call_noalloc(batch=0, parents=None, tokens=None, target_logits=None,
                        draft_logits=None, uniforms=None, accept_len=None, accepted_node=None,
                        bonus_token=None, status=None) == tv.TV_OK


def test_noalloc_scratch_covers_every_valid_size():
    """The static scratch (3 MiB) holds the workspace of the largest call the
    limits allow."""
    assert tv.tv_workspace_size(tv.TV_MAX_BATCH, tv.TV_MAX_NODES, tv.TV_MAX_VOCAB) <= 3 << 20


def call_stats(**kw):
    args = dict(batch=2, num_nodes=5, vocab=100, parents=A, tokens=A, target_logits=A,
                draft_logits=A + 0x1000, dtype=tv.TV_DTYPE_BF16, temperature=1.0, uniforms=A,
                mode=0, target_max=A, target_sum=A, draft_max=A, draft_sum=A, accept_len=A,
                accepted_node=A, bonus_token=A, status=A, workspace=WS,
                workspace_bytes=tv.tv_workspace_size(2, 5, 100))
    args.update(kw)
    return tv.tv_verify_stats(**args)


@pytest.mark.parametrize("kw,want", [
    (dict(batch=-1), tv.TV_ERR_INVALID_ARG),
    (dict(temperature=0.0), tv.TV_ERR_INVALID_ARG),
    (dict(parents=None), tv.TV_ERR_INVALID_ARG),
    (dict(target_max=None), tv.TV_ERR_INVALID_ARG),
    (dict(target_sum=None), tv.TV_ERR_INVALID_ARG),
    (dict(draft_max=None), tv.TV_ERR_INVALID_ARG),
    (dict(draft_sum=None), tv.TV_ERR_INVALID_ARG),
    (dict(target_sum=A + 4), tv.TV_ERR_INVALID_ARG),
    (dict(draft_max=A + 2), tv.TV_ERR_INVALID_ARG),
    (dict(workspace=None), tv.TV_ERR_WORKSPACE),
    (dict(num_nodes=tv.TV_MAX_NODES + 1), tv.TV_ERR_UNSUPPORTED),
])
def test_verify_stats_argument_errors_launch_nothing(kw, want):
    assert call_stats(**kw) == want


def test_verify_stats_empty_batch_is_ok():
    assert call_stats(batch=0, parents=None, tokens=None, target_logits=None, draft_logits=None,
                      uniforms=None, target_max=None, target_sum=None, draft_max=None,
                      draft_sum=None, accept_len=None, accepted_node=None, bonus_token=None,
                      status=None, workspace=None, workspace_bytes=0) == tv.TV_OK


def call_lmhead(**kw):
    args = dict(rows=4, hidden_size=64, vocab=1000, hidden=A, weight=A + 0x1000,
                temperature=1.0, logits=A, row_max=A, row_sum=A, workspace=WS,
                workspace_bytes=tv.tv_lmhead_workspace_size(4, 1000))
    args.update(kw)
    return tv.tv_lmhead_stats(**args)


@pytest.mark.parametrize("kw,want", [
    (dict(rows=-1), tv.TV_ERR_INVALID_ARG),
    (dict(hidden_size=4), tv.TV_ERR_INVALID_ARG),
    (dict(hidden_size=60), tv.TV_ERR_UNSUPPORTED),
    (dict(vocab=1), tv.TV_ERR_INVALID_ARG),
    (dict(vocab=tv.TV_MAX_VOCAB + 1), tv.TV_ERR_UNSUPPORTED),
    (dict(rows=tv.TV_MAX_LMHEAD_ROWS + 1), tv.TV_ERR_UNSUPPORTED),
    (dict(hidden_size=tv.TV_MAX_HIDDEN + 8), tv.TV_ERR_UNSUPPORTED),
    (dict(temperature=float("nan")), tv.TV_ERR_INVALID_ARG),
    (dict(temperature=1e-5), tv.TV_ERR_UNSUPPORTED),
    (dict(hidden=None), tv.TV_ERR_INVALID_ARG),
    (dict(weight=None), tv.TV_ERR_INVALID_ARG),
    (dict(logits=None), tv.TV_ERR_INVALID_ARG),
    (dict(row_max=None), tv.TV_ERR_INVALID_ARG),
    (dict(row_sum=None), tv.TV_ERR_INVALID_ARG),
    (dict(hidden=A + 8), tv.TV_ERR_INVALID_ARG),
    (dict(weight=A + 0x1008), tv.TV_ERR_INVALID_ARG),
    (dict(logits=A + 1), tv.TV_ERR_INVALID_ARG),
    (dict(row_sum=A + 4), tv.TV_ERR_INVALID_ARG),
    (dict(workspace=None), tv.TV_ERR_WORKSPACE),
    (dict(workspace=WS + 64), tv.TV_ERR_WORKSPACE),
    (dict(workspace_bytes=16), tv.TV_ERR_WORKSPACE),
])
def test_lmhead_argument_errors_launch_nothing(kw, want):
    assert call_lmhead(**kw) == want


def test_lmhead_empty_and_workspace_size():
    assert call_lmhead(rows=0, hidden=None, weight=None, logits=None, row_max=None,
                       row_sum=None, workspace=None, workspace_bytes=0) == tv.TV_OK
    assert tv.tv_lmhead_workspace_size(0, 1000) == 0
    assert tv.tv_lmhead_workspace_size(1, 1) == 0
    # one float maximum and one float sum per row and 256-column tile
    a = tv.tv_lmhead_workspace_size(16640, 128256)
    assert a % 256 == 0 and a >= 2 * 16640 * 501 * 4
