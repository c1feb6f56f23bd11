"""Monte-Carlo check of losslessness on the tiny exact-check workload: V = 8,
complete binary tree two levels deep, context-keyed target N(0, 2^2) and draft
target + N(0, 1) per context, temperature 1, seed 0. 10^5 seeded trials per
sibling mode; the padded first two output tokens (Lemma l1) and the first token
are compared with the target by chi-square (cells merged until each expects at
least 5). Passes if p > 1e-3 (fixed seeds, so the outcome is deterministic)."""

import multiprocessing as mp

import numpy as np
import pytest
from scipy import stats

import oracle.enumerate as E
import workloads as W
from oracle import (TREE_OK, WITH_REPLACEMENT, WITHOUT_REPLACEMENT, tempered_softmax,
                    verify_tree, verify_tree_tokenlevel)

TRIALS = 100_000
CHUNKS = 16


def _run_chunk(args):
    mode, verifier, chunk = args
    ver = verify_tree if verifier == "tv" else verify_tree_tokenlevel
    m = W.ContextModel(8, seed=0)
    par = W.binary_parents(2)
    rng = np.random.default_rng(np.random.SeedSequence([0, mode, chunk,
                                                        0 if verifier == "tv" else 1]))
    counts = np.zeros((8, 8), dtype=np.int64)
    for _ in range(TRIALS // CHUNKS):
        tok, zb, zs = W.draw_context_tree(rng, m, par, 1.0, mode)
        u = W.uniforms_np(rng, len(par))
        r = ver(par, tok, zb, zs, 1.0, u, mode)
        assert r.status == TREE_OK
        seq = list(E.path_tokens(par, tok, r.accepted_node)) + [r.bonus_token]
        while len(seq) < 2:
            p = tempered_softmax(m.target(tuple(seq)), 1.0)
            seq.append(int(rng.choice(8, p=p)))
        counts[seq[0], seq[1]] += 1
    return counts


def _chisq(counts, probs):
    counts = np.asarray(counts, dtype=np.float64).ravel()
    exp = np.asarray(probs, dtype=np.float64).ravel() * counts.sum()
    order = np.argsort(exp)
    c, e = counts[order], exp[order]
    # merge the smallest cells until every merged cell expects at least 5
    mc, me, acc_c, acc_e = [], [], 0.0, 0.0
    for ci, ei in zip(c, e):
        acc_c += ci
        acc_e += ei
        if acc_e >= 5:
            mc.append(acc_c)
            me.append(acc_e)
            acc_c = acc_e = 0.0
    if acc_e > 0:
        mc[-1] += acc_c
        me[-1] += acc_e
    return stats.chisquare(mc, me).pvalue


@pytest.mark.slow
@pytest.mark.parametrize("verifier", ["tv", "tokenlevel"])
@pytest.mark.parametrize("mode", [WITH_REPLACEMENT, WITHOUT_REPLACEMENT])
def test_monte_carlo_matches_target(mode, verifier):
    with mp.get_context("fork").Pool(8) as pool:
        parts = pool.map(_run_chunk, [(mode, verifier, c) for c in range(CHUNKS)])
    counts = sum(parts)
    m = W.ContextModel(8, seed=0)
    law = E.target_law(m, 1.0, 2)
    probs = np.zeros((8, 8))
    for (a, b), p in law.items():
        probs[a, b] = p
    assert counts.sum() == TRIALS
    p2 = _chisq(counts, probs)
    p1 = _chisq(counts.sum(axis=1), probs.sum(axis=1))
    assert p2 > 1e-3, p2
    assert p1 > 1e-3, p1
