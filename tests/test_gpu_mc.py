"""Losslessness of the HIP verifiers themselves (Theorem thm:TV_valid, via
Lemma l1): 10^5 draft trees of the tiny exact-check workload verified in one
launch per sibling mode and verifier, and the padded first two output tokens
compared with the target law by chi-square (needs an MI355X).

Workload: V = 8, complete binary tree two levels deep, context-keyed target
logits N(0, 2^2) and draft logits target + N(0, 1) per context (seed 0),
temperature 1. Children are drawn from the parent's draft distribution by
Gumbel-max (i.i.d.) or Gumbel-top-k (without replacement), matching the
sibling mode the verifier is told. The draws and uniforms use fixed seeds and
the launch is deterministic (one workgroup per tree at this vocabulary), so
the outcome is too; a test passes if p > 1e-3 for the pair and for the first
token."""

import numpy as np
import pytest
import torch

import oracle.enumerate as E
import paper_2505_12398_amd as tv
import parity
import workloads as W
from test_oracle_mc import _chisq

pytestmark = pytest.mark.gpu
DEV = "cuda"
TREES = 100_000
V = 8


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tv.load_library()
    yield


def _context_tables(m):
    """Target and draft rows of every context of length <= 2, as arrays
    indexed by the context's tokens."""
    t0, d0 = m.target(()), m.draft(())
    t1 = np.stack([m.target((a,)) for a in range(V)])
    d1 = np.stack([m.draft((a,)) for a in range(V)])
    t2 = np.stack([[m.target((a, c)) for c in range(V)] for a in range(V)])
    d2 = np.stack([[m.draft((a, c)) for c in range(V)] for a in range(V)])
    return t0, d0, t1, d1, t2, d2


def _draw_children(rng, zs_rows, mode):
    """Two children per tree from per-tree draft logit rows [B][V] (T = 1)."""
    B = zs_rows.shape[0]
    if mode == W.WITH_REPLACEMENT:
        a = np.argmax(zs_rows + W.gumbel_np(rng, (B, V)), axis=1)
        b = np.argmax(zs_rows + W.gumbel_np(rng, (B, V)), axis=1)
        return a, b
    order = np.argsort(-(zs_rows + W.gumbel_np(rng, (B, V))), axis=1, kind="stable")
    return order[:, 0], order[:, 1]


def _draw_batch(seed, mode):
    m = W.ContextModel(V, seed=0)
    t0, d0, t1, d1, t2, d2 = _context_tables(m)
    rng = np.random.default_rng(np.random.SeedSequence([seed, mode]))
    B = TREES
    x1, x2 = _draw_children(rng, np.tile(d0, (B, 1)), mode)       # nodes 1, 2
    x3, x4 = _draw_children(rng, d1[x1], mode)                     # children of node 1
    x5, x6 = _draw_children(rng, d1[x2], mode)                     # children of node 2
    tok = np.stack([np.zeros(B, np.int64), x1, x2, x3, x4, x5, x6], axis=1).astype(np.int32)
    zb = np.stack([np.tile(t0, (B, 1)), t1[x1], t1[x2], t2[x1, x3], t2[x1, x4], t2[x2, x5],
                   t2[x2, x6]], axis=1)
    zs = np.stack([np.tile(d0, (B, 1)), d1[x1], d1[x2], d2[x1, x3], d2[x1, x4], d2[x2, x5],
                   d2[x2, x6]], axis=1)
    u = W.uniforms_np(rng, (B, 7))
    par = np.tile(W.binary_parents(2), (B, 1))
    return m, rng, parity.from_numpy(par, tok, zb, zs, u, 1.0, mode, DEV)


@pytest.mark.parametrize("tokenlevel", [False, True])
@pytest.mark.parametrize("mode", [W.WITH_REPLACEMENT, W.WITHOUT_REPLACEMENT])
def test_gpu_output_law_is_the_target(mode, tokenlevel):
    m, rng, bt = _draw_batch(7 + int(tokenlevel), mode)
    out = tv.verify_batch(bt["parents"], bt["tokens"], bt["target"], bt["draft"], 1.0,
                          bt["uniforms"], mode, tokenlevel=tokenlevel, want_nodes=False,
                          want_counters=False)
    st = out.status.cpu().numpy()
    acc = out.accepted_node.cpu().numpy()
    y = out.bonus_token.cpu().numpy()
    assert (st == tv.TV_TREE_OK).all()
    tok = bt["tokens"].cpu().numpy()
    par = W.binary_parents(2)
    depth = W.node_depths(par)
    first = np.where(depth[acc] >= 1, tok[np.arange(TREES), np.where(acc >= 3, par[acc], acc)],
                     y)
    second = np.where(depth[acc] >= 2, tok[np.arange(TREES), acc],
                      np.where(depth[acc] == 1, y, -1))
    # tau = 0: the output is Y alone; pad it with a token from the target at (Y,)
    pad = np.nonzero(second < 0)[0]
    t1 = np.stack([m.target((a,)) for a in range(V)])
    p1 = np.exp(t1 - t1.max(axis=1, keepdims=True))
    p1 /= p1.sum(axis=1, keepdims=True)
    for i in pad:
        second[i] = rng.choice(V, p=p1[first[i]])
    counts = np.zeros((V, V), np.int64)
    np.add.at(counts, (first, second), 1)
    law = E.target_law(m, 1.0, 2)
    probs = np.zeros((V, V))
    for (a, b), p in law.items():
        probs[a, b] = p
    p2 = _chisq(counts, probs)
    p1v = _chisq(counts.sum(axis=1), probs.sum(axis=1))
    mean_tau = float(depth[acc].mean())
    print(f"mode={mode} tokenlevel={tokenlevel}: {TREES} trees, mean tau {mean_tau:.4f}, "
          f"chi-square p (pair) {p2:.3g}, p (first) {p1v:.3g}", flush=True)
    assert p2 > 1e-3, p2
    assert p1v > 1e-3, p1v
