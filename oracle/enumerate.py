"""Exact output laws of the oracle verifiers, by enumeration.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The losslessness theorem (Sec. 3.3, Theorem ``thm:TV_valid``) says the output
(X^tau, Y) of Traversal Verification is distributed as the target model. Lemma
``l1`` (App. A) restates it for a fixed maximum depth gamma_max: pad the output
with tokens drawn from the target until it has gamma_max tokens; the padded
sequence must then follow the target's autoregressive law. Here the padding goes
one token further (length gamma_max + 1) so that Y after a full-depth leaf is
covered too.

Two layers of enumeration:

* :func:`decision_branches` runs a verifier under every combination of
  accept/reject outcomes, weighting each run by the product of theta or
  1 - theta over its tests (deterministic tests, theta in {0, 1}, do not branch);
* :func:`draft_tree_law` sums over every draft tree a context-keyed model can
  produce (Def. ``de_tree``: each node's children drawn from the draft
  distribution at that node, i.i.d. or without replacement), weighting each
  tree by its sampling probability.
"""

from __future__ import annotations

from collections import defaultdict

import numpy as np

from .tv_oracle import (TREE_OK, WITHOUT_REPLACEMENT, WITH_REPLACEMENT,
                        tempered_softmax, verify_tree)


class _NewDecision(Exception):
    pass


def decision_branches(run):
    """All outcomes of ``run(decide)``: a list of (probability, result)."""
    out = []
    scripts = [()]
    while scripts:
        script = scripts.pop()
        state = {"pos": 0, "w": 1.0}

        def decide(node, theta, script=script, state=state):
            if theta >= 1.0:
                return True
            if theta <= 0.0:
                return False
            pos = state["pos"]
            if pos < len(script):
                choice = script[pos]
                state["pos"] = pos + 1
                state["w"] *= theta if choice else (1.0 - theta)
                return choice
            raise _NewDecision()

        try:
            res = run(decide)
        except _NewDecision:
            scripts.append(script + (True,))
            scripts.append(script + (False,))
            continue
        out.append((state["w"], res))
    return out


def path_tokens(parents, tokens, node):
    """Drafted tokens on the path root..node, root excluded, in order."""
    seq = []
    while node > 0:
        seq.append(int(tokens[node]))
        node = int(parents[node])
    return tuple(reversed(seq))


def fixed_tree_law(verifier, parents, tokens, zb, zs, T, mode):
    """Exact law of (X^tau, Y) for one fixed tree: {token tuple: probability},
    the tuple being the accepted drafted tokens followed by Y."""
    law = defaultdict(float)
    branches = decision_branches(
        lambda d: verifier(parents, tokens, zb, zs, T, None, mode, decide=d))
    for w, res in branches:
        if res.status != TREE_OK:
            raise ValueError(f"verifier returned status {res.status}")
        prefix = path_tokens(parents, tokens, res.accepted_node)
        for y, py in enumerate(res.y_weights):
            if py > 0.0:
                law[prefix + (y,)] += w * py
    return dict(law)


def _contexts(parents, tokens):
    return [path_tokens(parents, tokens, i) for i in range(len(parents))]


def _draft_trees(parents, model, T, sampling):
    """Every token assignment of the tree shape with its probability under the
    model's tempered draft distributions. ``sampling`` is WITH_REPLACEMENT
    (children i.i.d.) or WITHOUT_REPLACEMENT (siblings drawn one after another,
    each from the draft with the earlier siblings removed)."""
    n1 = len(parents)
    V = model.vocab

    def rec(i, tokens, prob):
        if i == n1:
            yield list(tokens), prob
            return
        j = int(parents[i])
        q = tempered_softmax(model.draft(path_tokens(parents, tokens, j)), T)
        earlier = [int(tokens[c]) for c in range(1, i) if int(parents[c]) == j]
        if sampling == WITHOUT_REPLACEMENT:
            free = 1.0 - sum(q[x] for x in earlier)
        for x in range(V):
            if sampling == WITHOUT_REPLACEMENT:
                if x in earlier:
                    continue
                px = q[x] / free
            else:
                px = q[x]
            if px == 0.0:
                continue
            tokens[i] = x
            yield from rec(i + 1, tokens, prob * px)
        tokens[i] = 0

    yield from rec(1, [0] * n1, 1.0)


def tree_rows(parents, tokens, model):
    """Per-node target and draft logit rows of a tree under a context model."""
    ctx = _contexts(parents, tokens)
    zb = np.stack([model.target(c) for c in ctx])
    zs = np.stack([model.draft(c) for c in ctx])
    return zb, zs


def padded_law(out_law, model, T, length):
    """Pad every output sequence with target draws up to ``length`` tokens."""
    padded = defaultdict(float)
    stack = [(seq, p) for seq, p in out_law.items()]
    while stack:
        seq, p = stack.pop()
        if len(seq) >= length:
            padded[seq[:length]] += p
            continue
        nxt = tempered_softmax(model.target(seq), T)
        for x, px in enumerate(nxt):
            if px > 0.0:
                stack.append((seq + (x,), p * px))
    return dict(padded)


def target_law(model, T, length):
    """The target model's law of the next ``length`` tokens after the root,
    the right-hand side of Eq. (e7-5)."""
    return padded_law({(): 1.0}, model, T, length)


def draft_tree_law(verifier, parents, model, T, sampling, verify_mode, length=None):
    """Exact law of the padded output of ``verifier`` over all draft trees of the
    given shape drawn from ``model``. ``length`` defaults to gamma_max + 1."""
    depth = [0] * len(parents)
    for i in range(1, len(parents)):
        depth[i] = depth[int(parents[i])] + 1
    if length is None:
        length = max(depth) + 1
    total = defaultdict(float)
    for tokens, ptree in _draft_trees(parents, model, T, sampling):
        zb, zs = tree_rows(parents, tokens, model)
        law = fixed_tree_law(verifier, parents, tokens, zb, zs, T, verify_mode)
        for seq, p in padded_law(law, model, T, length).items():
            total[seq] += ptree * p
    return dict(total)


def law_distance(a, b):
    """Largest absolute difference between two laws over the union of cells."""
    keys = set(a) | set(b)
    return max(abs(a.get(k, 0.0) - b.get(k, 0.0)) for k in keys)


def expected_accept_len(verifier, parents, tokens, zb, zs, T, mode):
    """E[tau] for one fixed tree, by decision enumeration."""
    return sum(w * res.accept_len for w, res in decision_branches(
        lambda d: verifier(parents, tokens, zb, zs, T, None, mode, decide=d)))


__all__ = ["decision_branches", "fixed_tree_law", "draft_tree_law", "padded_law",
           "target_law", "law_distance", "tree_rows", "path_tokens",
           "expected_accept_len", "verify_tree", "WITH_REPLACEMENT",
           "WITHOUT_REPLACEMENT"]
