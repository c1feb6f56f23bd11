"""Pins for the CPU oracle: checks against what the paper and the mathematics
fix, never against the oracle itself. Each pin raises AssertionError when
violated. tests/test_oracle_pins.py runs them on the oracle as written;
tests/test_oracle_mutations.py plants plausible mistakes in the oracle and
checks that some pin fails.

All calls go through module attributes (``O.verify_tree``) so that a planted
mistake in one step is seen by every pin.
"""

from __future__ import annotations

import json
import os
from fractions import Fraction

import numpy as np

import oracle.tv_oracle as O
import oracle.enumerate as E
import oracle.draft_sampler as DS
import oracle.lmhead as LM
import workloads as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
ALMOST_ONE = np.float32(1.0 - 2.0 ** -24)     # rejects any theta < 1


def golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def frac(v):
    return float(Fraction(v[0], v[1]))


def _close(a, b, tol=1e-12, what=""):
    assert abs(float(a) - float(b)) <= tol, f"{what}: {a!r} != {b!r}"


def _single_node_rows(target, draft, n1):
    zb = np.tile(np.log(np.asarray(target, dtype=np.float64)), (n1, 1))
    zs = np.tile(np.log(np.asarray(draft, dtype=np.float64)), (n1, 1))
    return zb, zs


# ---------------------------------------------------------------------------
# Values the paper prints
# ---------------------------------------------------------------------------

def pin_worked_example_trace():
    """Sec. 3.2: traversal order, chain rates and the parent update numbers,
    following every rejection (all uniforms just below 1)."""
    g = golden("worked_example.json")
    par, tok, zb, zs, T = W.worked_example()
    u = np.full(6, ALMOST_ONE, np.float32)
    u[0] = 0.5
    r = O.verify_tree(par, tok, zb, zs, T, u, O.WITHOUT_REPLACEMENT)
    assert r.status == O.TREE_OK
    assert r.test_order == g["traversal_order"], r.test_order
    pr = g["printed"]
    tol = g["printed_tolerance"]
    _close(r.node_theta[3], pr["accept_chain_X1X3_traversal"], tol, "theta X3 printed")
    # theta(X4) = p'(X1) * b'(c)/s'(c) with b' = [0,0,1] and s'(c) = 1/7 (Eq. e1, e2)
    _close(r.node_theta[4] / 7.0, pr["p_prime_X1_after_X3"], tol, "p' X1 printed")
    _close(r.node_theta[4], pr["accept_chain_X1X4"], tol, "theta X4 printed")
    _close(r.node_theta[1], pr["p_prime_X1_after_X4"], 0.0, "p' X1 -> 0")
    ex = g["exact_readings"]
    for node, key in [(1, "p_ini_X1"), (3, "p_ini_X3")]:
        _close(r.p_init[node], frac(ex[key]), 1e-12, key)
    for node, key in [(3, "theta_X3"), (4, "theta_X4"), (1, "theta_X1"), (5, "theta_X5"),
                      (2, "theta_X2")]:
        _close(r.node_theta[node], frac(ex[key]), 1e-12, key)
    assert r.accepted_node == 2 and r.accept_len == 1
    # Y comes from X2's residual after X5 (token a) is rejected: [0, 1/3, 2/3].
    _close(r.y_weights[0], 0.0, 0.0, "residual a")
    _close(r.y_weights[1], 1 / 3, 1e-12, "residual b")


def pin_worked_example_tokenlevel():
    """Sec. 3.2: token-level acceptance of chain X1X3 is 0.5 (X1 at 1/2, X3 sure)."""
    g = golden("worked_example.json")
    par, tok, zb, zs, T = W.worked_example()
    law = {}
    for w, res in E.decision_branches(
            lambda d: O.verify_tree_tokenlevel(par, tok, zb, zs, T, None,
                                               O.WITHOUT_REPLACEMENT, decide=d)):
        law[res.accepted_node] = law.get(res.accepted_node, 0.0) + w
    _close(law.get(3, 0.0), g["printed"]["accept_chain_X1X3_tokenlevel"], 1e-12, "TL X1X3")


def pin_worked_example_law():
    """Exact accept law of both verifiers on the Sec. 3.2 tree (products of the
    printed steps)."""
    g = golden("worked_example.json")["derived_law"]
    par, tok, zb, zs, T = W.worked_example()
    for ver, key, tkey in [(O.verify_tree, "traversal_accepted_node", "traversal_expected_tau"),
                           (O.verify_tree_tokenlevel, "tokenlevel_accepted_node",
                            "tokenlevel_expected_tau")]:
        law = {}
        etau = 0.0
        for w, res in E.decision_branches(
                lambda d: ver(par, tok, zb, zs, T, None, O.WITHOUT_REPLACEMENT, decide=d)):
            law[res.accepted_node] = law.get(res.accepted_node, 0.0) + w
            etau += w * res.accept_len
        want = {int(k): frac(v) for k, v in g[key].items()}
        assert set(law) == set(want), (key, law)
        for k, v in want.items():
            _close(law[k], v, 1e-12, f"{key}[{k}]")
        _close(etau, frac(g[tkey]), 1e-12, tkey)


def pin_single_token_table1():
    """Sec. 2.1 Table 1: acceptance probability of each drafted token, the
    residual after rejecting a, and an output law equal to the target."""
    g = golden("single_token.json")
    par = np.array([-1, 0], np.int32)
    zb, zs = _single_node_rows(g["target"], g["draft"], 2)
    resid = np.asarray(g["residual_unnormalised"], dtype=np.float64)
    np.testing.assert_allclose(resid / resid.sum(), [frac(v) for v in g["residual"]],
                               atol=1e-12)
    first = np.zeros(3)
    for x, name in enumerate("abc"):
        tok = np.array([0, x], np.int32)
        acc = 0.0
        for w, res in E.decision_branches(
                lambda d: O.verify_tree(par, tok, zb, zs, 1.0, None, O.WITHOUT_REPLACEMENT,
                                        decide=d)):
            if res.accepted_node == 1:
                acc += w
            else:   # rejected: Y from the normalised residual [M_b - M_s]_+
                assert res.accepted_node == 0
                np.testing.assert_allclose(res.y_weights, resid / resid.sum(), atol=1e-12)
        _close(acc, g["accept_prob"][name], 1e-12, f"accept {name}")
        law = E.fixed_tree_law(O.verify_tree, par, tok, zb, zs, 1.0, O.WITHOUT_REPLACEMENT)
        for seq, p in law.items():
            first[seq[0]] += g["draft"][x] * p
    # Drafting x with M_s(x) and verifying: the first output token follows M_b.
    np.testing.assert_allclose(first, g["target"], atol=1e-12)


def pin_rrsw_example():
    """Sec. 2.2: after rejecting a, residual [0,1/3,2/3], draft [0,3/4,1/4], and a
    second candidate b is accepted with probability 4/9 (c with certainty).
    A root with two leaf children: both verifiers coincide here."""
    g = golden("rrsw_example.json")
    par = np.array([-1, 0, 0], np.int32)
    zb, zs = _single_node_rows(g["target"], g["draft"], 3)
    for second, key in [(1, "b"), (2, "c")]:
        tok = np.array([0, 0, second], np.int32)
        u = np.array([0.5, ALMOST_ONE, 0.5], np.float32)
        for ver in (O.verify_tree, O.verify_tree_tokenlevel):
            r = ver(par, tok, zb, zs, 1.0, u, O.WITHOUT_REPLACEMENT)
            _close(r.node_theta[1], 0.5, 1e-12, "first candidate")
            _close(r.node_theta[2], frac(g["accept_prob_second_candidate"][key]), 1e-12,
                   f"second candidate {key}")
    # Residual after rejecting both a and b: Y's distribution at the root.
    tok = np.array([0, 0, 1], np.int32)
    u = np.array([0.5, ALMOST_ONE, ALMOST_ONE], np.float32)
    r = O.verify_tree_tokenlevel(par, tok, zb, zs, 1.0, u, O.WITHOUT_REPLACEMENT)
    res_a = np.array([frac(v) for v in g["after_rejecting_a"]["residual_target"]])
    drf_a = np.array([frac(v) for v in g["after_rejecting_a"]["draft_without_a"]])
    want = np.maximum(res_a - drf_a, 0)
    np.testing.assert_allclose(r.y_weights, want / want.sum(), atol=1e-12)


# ---------------------------------------------------------------------------
# Mathematics the paper fixes
# ---------------------------------------------------------------------------

def pin_tempered_softmax_inverse():
    """softmax(T * log p / T) = p for any T > 0 (temperature undoes its own
    scaling), and the largest logit keeps the largest probability."""
    rng = np.random.default_rng(7)
    p = rng.dirichlet(np.ones(11))
    for T in (0.7, 1.0, 1.9):
        q = O.tempered_softmax(T * np.log(p), np.float32(T))
        np.testing.assert_allclose(q, p, rtol=1e-6, atol=1e-12)
    z = rng.normal(size=9)
    a = O.tempered_softmax(z, np.float32(0.5))
    b = O.tempered_softmax(z, np.float32(2.0))
    assert a.max() > b.max()    # lower temperature sharpens


def pin_inverse_cdf_law():
    """The final sample has law w / sum(w): over the 2^12 grid of uniforms
    u = k / 2^12 each token's count is its weight times 2^12 up to one."""
    w = np.array([0.0, 3.0, 1.0, 0.0, 4.0, 0.5, 0.0, 7.5])
    n = 2 ** 12
    counts = np.zeros(len(w))
    for k in range(n):
        y, _ = O.inverse_cdf(w, k / n)
        counts[y] += 1
    want = w / w.sum() * n
    assert np.all(np.abs(counts - want) <= 1.0), (counts, want)
    assert counts[w == 0].sum() == 0


def pin_lossless_exact():
    """Theorem thm:TV_valid via Lemma l1: the padded output law equals the
    target law, over all draft trees of a tiny context model, in both matched
    sibling modes, for Traversal Verification and the token-level baseline."""
    m = W.ContextModel(3, seed=0)
    par = W.binary_parents(2)
    tl = E.target_law(m, 1.0, 3)
    for ver in (O.verify_tree, O.verify_tree_tokenlevel):
        for mode in (O.WITH_REPLACEMENT, O.WITHOUT_REPLACEMENT):
            law = E.draft_tree_law(ver, par, m, 1.0, mode, mode)
            d = E.law_distance(law, tl)
            assert d < 1e-12, (ver.__name__, mode, d)


def pin_lossless_irregular_T07():
    """Same check on an irregular tree (3 children at the root, 2 below the
    first) at temperature 0.7, V = 4."""
    m = W.ContextModel(4, seed=3)
    par = np.array([-1, 0, 0, 0, 1, 1], np.int32)
    T = np.float32(0.7)
    tl = E.target_law(m, T, 3)
    for mode in (O.WITH_REPLACEMENT, O.WITHOUT_REPLACEMENT):
        law = E.draft_tree_law(O.verify_tree, par, m, T, mode, mode)
        d = E.law_distance(law, tl)
        assert d < 1e-12, (mode, d)


def pin_chain_optimality():
    """Theorem thm:chain_op and App. B: on a chain, E[tau] equals the draft
    expectation of sum_l p^ini(alpha_l), and P(tau >= l | X^l = alpha^l) equals
    p^ini(alpha_l); the token-level verifier does not do better."""
    V, depth = 3, 3
    m = W.ContextModel(V, seed=5)
    par = W.chain_parents(depth)
    e_tv = e_tl = e_pini = 0.0
    ge = {}      # (prefix) -> [sum P(tree) P(tau >= l), sum P(tree) p_ini]
    for tokens, ptree in E._draft_trees(par, m, 1.0, O.WITH_REPLACEMENT):
        zb, zs = E.tree_rows(par, tokens, m)
        br = E.decision_branches(
            lambda d: O.verify_tree(par, tokens, zb, zs, 1.0, None, O.WITH_REPLACEMENT,
                                    decide=d))
        e_tv += ptree * sum(w * r.accept_len for w, r in br)
        e_tl += ptree * E.expected_accept_len(O.verify_tree_tokenlevel, par, tokens, zb, zs,
                                              1.0, O.WITH_REPLACEMENT)
        pini = br[0][1].p_init
        e_pini += ptree * float(pini[1:].sum())
        for l in range(1, depth + 1):
            key = tuple(tokens[1:l + 1])
            acc = ge.setdefault(key, [0.0, 0.0])
            acc[0] += ptree * sum(w for w, r in br if r.accept_len >= l)
            acc[1] += ptree * pini[l]
    assert abs(e_tv - e_pini) < 1e-12, (e_tv, e_pini)
    assert e_tv >= e_tl - 1e-12, (e_tv, e_tl)
    for key, (a, b) in ge.items():
        assert abs(a - b) < 1e-12, (key, a, b)


def pin_identical_models():
    """M_s = M_b: every chain rate is 1, so the first leaf is accepted at once
    and Y comes from that leaf's target row."""
    rng = np.random.default_rng(11)
    par = W.binary_parents(3)
    n1, V = len(par), 17
    z = rng.normal(0, 2, (n1, V))
    tok = rng.integers(0, V, n1).astype(np.int32)
    u = W.uniforms_np(rng, n1)
    r = O.verify_tree(par, tok, z, z.copy(), 1.0, u, O.WITH_REPLACEMENT)
    assert r.status == O.TREE_OK
    assert np.all(r.p_init == 1.0)
    assert r.accepted_node == 7 and r.test_order == [7]
    np.testing.assert_allclose(r.y_weights, O.tempered_softmax(z[7], 1.0), atol=0)


def pin_depth1_equals_rrsw():
    """A root with leaf children only: p(root) = 1 makes Eq. (e1)-(e3) reduce to
    Algorithm 2, so both verifiers give identical decisions, thresholds and Y."""
    rng = np.random.default_rng(12)
    for trial in range(40):
        V = 50
        k = int(rng.integers(1, 6))
        par = np.array([-1] + [0] * k, np.int32)
        zb = rng.normal(0, 2, (k + 1, V))
        zs = zb + rng.normal(0, 1, (k + 1, V))
        mode = int(trial % 2)
        tok = np.concatenate([[0], rng.choice(V, k, replace=mode == O.WITH_REPLACEMENT)]) \
            .astype(np.int32)
        u = W.uniforms_np(rng, k + 1)
        a = O.verify_tree(par, tok, zb, zs, 1.0, u, mode)
        b = O.verify_tree_tokenlevel(par, tok, zb, zs, 1.0, u, mode)
        assert a.accepted_node == b.accepted_node and a.bonus_token == b.bonus_token
        assert a.test_order == b.test_order
        assert np.array_equal(a.node_theta, b.node_theta)


def pin_invariants():
    """Along random traversals: 0 <= p' <= p at every update (Eq. e3 with
    S <= p), the residual sums to one and is zero on the rejected token (Eq. e1),
    and the draft update keeps a distribution (Eq. e2)."""
    rng = np.random.default_rng(13)
    V = 40
    for _ in range(200):
        b = rng.dirichlet(np.ones(V))
        s = rng.dirichlet(np.ones(V))
        p = float(rng.uniform(0.05, 1.0))
        x = int(np.argmax(s / b))            # a token with p*b(x) < s(x)
        d, S = O.residual_e1(p, b, s)
        assert S <= p + 1e-15
        if S == 0.0:     # p*b <= s everywhere: the parent can no longer be accepted
            assert np.all(p * b <= s)
            continue
        pn = O.acceptance_update_e3(S, p)
        assert 0.0 <= pn <= p + 1e-15
        bn = d / S
        assert abs(bn.sum() - 1.0) < 1e-12 and bn[x] == 0.0
        sn = O.draft_update_e2(s, x)
        assert sn[x] == 0.0 and abs(sn.sum() - 1.0) < 1e-12


def pin_early_rejection_worked_example():
    """Sec. 3.2 with every drafted node rejected: after X4, the last child of X1,
    is rejected, p(X1) = 1/11 <= u, and X1 is then rejected (its rate falls to
    0): that update is the one an early-rejecting verifier skips. After X5, the
    only child of X2, p(X2) = 1 > u and X2 is accepted: that update is needed
    (it gives Y's residual). Updates after X3 (X4 still remains) and at the root
    never qualify."""
    par, tok, zb, zs, T = W.worked_example()
    u = np.full(6, ALMOST_ONE, np.float32)
    u[0] = 0.5
    r = O.verify_tree(par, tok, zb, zs, T, u, O.WITHOUT_REPLACEMENT)
    assert r.residual_passes == 4, r.residual_passes      # after X3, X4, X1, X5
    assert r.early_nodes == [1], r.early_nodes
    assert r.counters_early[1] == 3
    # the rule's checks: u(X1) - 1/11 and 1 - u(X2) = 2^-24
    _close(r.early_margin, 2.0 ** -24, 1e-18, "early margin")
    # X1 tested with u just above its rate: not skipped, same decisions
    u[1] = np.float32(1.0 / 11.0) * np.float32(0.5)
    r2 = O.verify_tree(par, tok, zb, zs, T, u, O.WITHOUT_REPLACEMENT)
    assert r2.early_nodes == [] and r2.test_order == r.test_order


def pin_early_rejection_sound():
    """Every update counted as skippable is followed by the rejection of its
    node with theta <= u (p never rises under Eq. e3), on random irregular trees
    in both sibling modes; and such updates occur."""
    rng = np.random.default_rng(21)
    seen = 0
    for t in range(120):
        V = int(rng.integers(3, 12))
        par = W.geometric_bfs_parents(rng, 12, 4)
        n1 = len(par)
        zb = rng.normal(0.0, 2.0, (n1, V))
        zs = zb + rng.normal(0.0, 1.5, (n1, V))
        mode = O.WITHOUT_REPLACEMENT if t % 2 == 0 else O.WITH_REPLACEMENT
        tok = np.zeros(n1, np.int64)
        for j in range(n1):
            kids = [i for i in range(n1) if par[i] == j]
            if kids:
                q = np.exp(zs[j] - zs[j].max())
                q /= q.sum()
                pick = rng.choice(V, size=len(kids), replace=(mode == O.WITH_REPLACEMENT
                                                              or len(kids) > V), p=q)
                tok[kids] = pick
        u = (rng.integers(0, 2 ** 24, n1) * 2.0 ** -24).astype(np.float32)
        r = O.verify_tree(par, tok, zb, zs, 1.0, u, mode)
        if r.status != O.TREE_OK:
            continue
        for j in r.early_nodes:
            seen += 1
            assert j != 0
            assert r.node_state[j] == O.NODE_REJECTED, (t, j)
            assert r.node_theta[j] <= float(u[j]), (t, j, r.node_theta[j], u[j])
        assert r.counters_early[1] == r.residual_passes - len(r.early_nodes)
    assert seen > 20, seen


def pin_draft_sampler_law():
    """Def. de_tree: two children of the root drawn from the tempered Table 1
    draft [.6, .3, .1] at T = 0.7. Over a 200 x 200 grid of uniforms the joint
    frequency of the two tokens matches q(x1) q(x2) / (1 - q(x1)) without
    replacement and q(x1) q(x2) with replacement (each inverse-CDF interval is
    matched to within one grid step, so 3/200 bounds the error)."""
    q0 = np.array([0.6, 0.3, 0.1])
    T = 0.7
    q = q0 ** (1.0 / np.float64(np.float32(T)))
    q /= q.sum()
    zs = np.tile(np.log(q0), (3, 1))
    par = np.array([-1, 0, 0])
    M = 200
    grid = (np.arange(M) + 0.5) / M
    for mode in (O.WITHOUT_REPLACEMENT, O.WITH_REPLACEMENT):
        f = np.zeros((3, 3))
        for u1 in grid:
            for u2 in grid:
                r = DS.draw_tree_tokens(par, zs, T, np.array([0.5, u1, u2]), mode)
                assert r.status == O.TREE_OK and r.tokens[0] == -1
                f[r.tokens[1], r.tokens[2]] += 1.0 / (M * M)
        for a in range(3):
            for b in range(3):
                if mode == O.WITHOUT_REPLACEMENT:
                    want = 0.0 if a == b else q[a] * q[b] / (1.0 - q[a])
                else:
                    want = q[a] * q[b]
                assert abs(f[a, b] - want) <= 3.0 / M, (mode, a, b, f[a, b], want)


def pin_draft_sampler_statuses():
    """Error cases of the sampler: a parent link that does not point backwards,
    a NaN in a row with children, and more children than tokens without
    replacement (fine with replacement)."""
    zs = np.zeros((4, 2))
    u = np.full(4, 0.5)
    r = DS.draw_tree_tokens(np.array([-1, 0, 3, 1]), zs, 1.0, u)
    assert r.status == O.TREE_BAD_PARENT and np.all(r.tokens == -1)
    bad = zs.copy()
    bad[0, 1] = np.nan
    r = DS.draw_tree_tokens(np.array([-1, 0, 0, 0]), bad, 1.0, u)
    assert r.status == O.TREE_NONFINITE
    r = DS.draw_tree_tokens(np.array([-1, 0, 0, 0]), zs, 1.0, u, O.WITHOUT_REPLACEMENT)
    assert r.status == O.TREE_DEGENERATE
    r = DS.draw_tree_tokens(np.array([-1, 0, 0, 0]), zs, 1.0, u, O.WITH_REPLACEMENT)
    assert r.status == O.TREE_OK and list(r.tokens) == [-1, 1, 1, 1]
    # a NaN row and a row with too many siblings: the larger code (DEGENERATE)
    mixed = zs.copy()
    mixed[0, 0] = np.nan
    r = DS.draw_tree_tokens(np.array([-1, 0, 1, 1, 1]), np.vstack([mixed, zs[:1]]), 1.0,
                            np.full(5, 0.5), O.WITHOUT_REPLACEMENT)
    assert r.status == O.TREE_DEGENERATE and np.all(r.tokens == -1)
    # two children at V = 2 without replacement take both tokens
    r = DS.draw_tree_tokens(np.array([-1, 0, 0, 1]), zs, 1.0, u, O.WITHOUT_REPLACEMENT)
    assert r.status == O.TREE_OK and sorted(r.tokens[1:3]) == [0, 1]


def pin_committed_sequence():
    """Def. def2 on the Sec. 3.2 tree (X1..X5 drafted tokens a, c, b, c, a):
    accepting X4 outputs the chain X1 X4, tokens a c, then Y; accepting X2
    outputs c then Y; accepting the root outputs Y alone. The chain has as many
    nodes as the accepted node's depth."""
    g = golden("worked_example.json")
    par = g["parents"]
    voc = {t: i for i, t in enumerate(g["vocab"])}
    tok = [-1] + [voc[t] for t in g["tokens_X1_to_X5"]]
    assert O.committed_sequence(par, tok, 4, 2) == ([1, 4], [voc["a"], voc["c"], 2])
    assert O.committed_sequence(par, tok, 2, 0) == ([2], [voc["c"], 0])
    assert O.committed_sequence(par, tok, 0, 1) == ([], [1])
    rng = np.random.default_rng(5)
    for _ in range(50):
        p = W.geometric_bfs_parents(rng, 20, 5)
        a = int(rng.integers(0, len(p)))
        nodes, toks = O.committed_sequence(p, np.arange(len(p)), a, 7)
        assert len(nodes) == W.node_depths(p)[a] and toks[-1] == 7
        assert all(int(p[nodes[i + 1]]) == nodes[i] for i in range(len(nodes) - 1))
        assert not nodes or int(p[nodes[0]]) == 0


# ---------------------------------------------------------------------------
# Bookkeeping the kernels report: work counters, input widening, statuses
# ---------------------------------------------------------------------------

def pin_counters_worked_example():
    """Work counters on the Sec. 3.2 tree, derived by hand from their
    definitions: rows consulted = internal nodes that are proper ancestors of
    a tested node; residual updates = rejections followed by Eq. (e1)-(e3);
    leaf accepted = the accepted node has no children; tests = nodes compared
    with their uniform.

    * Every drafted node rejected (uniforms just below 1): tests X3, X4, X1,
      X5, X2 (X2's rate is 1, so it is accepted); their proper ancestors are
      X0, X1, X2; updates after X3, X4 (at X1), X1 (at X0) and X5 (at X2):
      (3, 4, 0, 5).
    * All uniforms 0: X3 (rate 2/3) is accepted at once; ancestors X0, X1; a
      leaf: (2, 0, 1, 1).
    * Token-level, every candidate rejected: X1 (1/2) rejected, update at X0;
      X2 (rate 1 on the residual) accepted; X5 (1/2) rejected, update at X2; Y
      from X2's residual. Tested X1, X2, X5 with ancestors X0, X2: (2, 2, 0, 3).
    * Token-level, all uniforms 0: X1 then X3 (rate 1) accepted; a leaf:
      (2, 0, 1, 2)."""
    par, tok, zb, zs, T = W.worked_example()
    hi = np.full(6, ALMOST_ONE, np.float32)
    hi[0] = 0.5
    lo = np.zeros(6, np.float32)
    cases = [(O.verify_tree, hi, (3, 4, 0, 5)), (O.verify_tree, lo, (2, 0, 1, 1)),
             (O.verify_tree_tokenlevel, hi, (2, 2, 0, 3)),
             (O.verify_tree_tokenlevel, lo, (2, 0, 1, 2))]
    for ver, u, want in cases:
        r = ver(par, tok, zb, zs, T, u, O.WITHOUT_REPLACEMENT)
        assert r.status == O.TREE_OK
        assert tuple(r.counters) == want, (ver.__name__, tuple(r.counters), want)


def pin_counters_identical_models():
    """M_s = M_b on a complete binary tree of depth 3: the first leaf (node 7)
    is accepted with rate 1 after no update; its proper ancestors 0, 1, 3 are
    the rows consulted: counters (3, 0, 1, 1). The token-level verifier
    accepts 1, 3, 7 in turn: (3, 0, 1, 3)."""
    rng = np.random.default_rng(11)
    par = W.binary_parents(3)
    n1, V = len(par), 17
    z = rng.normal(0, 2, (n1, V))
    tok = rng.integers(0, V, n1).astype(np.int32)
    u = W.uniforms_np(rng, n1)
    r = O.verify_tree(par, tok, z, z.copy(), 1.0, u, O.WITH_REPLACEMENT)
    assert tuple(r.counters) == (3, 0, 1, 1), tuple(r.counters)
    r = O.verify_tree_tokenlevel(par, tok, z, z.copy(), 1.0, u, O.WITH_REPLACEMENT)
    assert r.accepted_node == 7 and tuple(r.counters) == (3, 0, 1, 3), tuple(r.counters)


def pin_bf16_widening():
    """bfloat16 logits arrive as 16-bit patterns: the top half of an IEEE
    float32. All 65536 patterns widen to what torch's own bfloat16 -> float32
    conversion gives (NaN patterns to NaN), and a few values follow from the
    format by hand: 0x3FC0 = 1.5, 0xC000 = -2, 0x7F80 = +inf, 0xFF80 = -inf,
    0x0001 = 2^-133 (the smallest subnormal), 0x0080 = 2^-126."""
    import torch
    bits = np.arange(65536, dtype=np.uint16)
    got = O.to_f64(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).float().double().numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    hand = {0x3FC0: 1.5, 0xC000: -2.0, 0x7F80: np.inf, 0xFF80: -np.inf,
            0x0001: 2.0 ** -133, 0x0080: 2.0 ** -126, 0x0000: 0.0}
    for b, v in hand.items():
        assert O.to_f64(np.array([b], np.uint16))[0] == v, (hex(b), v)
    # float32 rows are widened as they are
    f = np.array([0.1, -3.5, 1e-40], np.float32)
    assert np.array_equal(O.to_f64(f), f.astype(np.float64))


def pin_verifier_statuses():
    """Per-tree statuses of both verifiers on hand-made cases: a root whose
    parent is not -1 or a link that does not point to an earlier node
    (BAD_PARENT, before token checks), a drafted token outside [0, V)
    (BAD_TOKEN), two siblings with one token without replacement (DUP_SIBLING;
    fine with replacement), a NaN, +inf or all--inf row with children and a
    drafted token whose draft logit is -inf (NONFINITE). Rows the verifier
    never reads (a leaf's draft row, a rejected leaf's target row) may hold
    anything."""
    par, tok, zb, zs, T = W.worked_example()
    u = np.full(6, ALMOST_ONE, np.float32)
    u[0] = 0.5
    W_ = O.WITHOUT_REPLACEMENT
    for ver in (O.verify_tree, O.verify_tree_tokenlevel):
        def st(p=par, t=tok, b=zb, s=zs, mode=W_):
            return ver(np.asarray(p), np.asarray(t), b, s, T, u, mode).status
        base = ver(par, tok, zb, zs, T, u, W_)
        assert base.status == O.TREE_OK
        assert st(p=[0, 0, 0, 1, 1, 2]) == O.TREE_BAD_PARENT
        assert st(p=[-1, 0, 0, 3, 1, 2]) == O.TREE_BAD_PARENT
        assert st(p=[-1, 0, 0, 1, 1, -1]) == O.TREE_BAD_PARENT
        assert st(p=[-1, 0, 0, 3, 1, 2], t=[0, 0, 2, 1, 2, 7]) == O.TREE_BAD_PARENT
        assert st(t=[0, 0, 2, 1, 2, 3]) == O.TREE_BAD_TOKEN
        assert st(t=[0, -1, 2, 1, 2, 0]) == O.TREE_BAD_TOKEN
        assert st(t=[5, 0, 2, 1, 2, 0]) == O.TREE_OK          # the root's token is unused
        assert st(t=[0, 0, 2, 1, 1, 0]) == O.TREE_DUP_SIBLING  # X3 and X4 both b
        assert st(t=[0, 0, 2, 1, 1, 0], mode=O.WITH_REPLACEMENT) == O.TREE_OK
        for bad in (np.nan, np.inf):
            for rows, which in ((zb, "target"), (zs, "draft")):
                z = rows.copy()
                z[0, 1] = bad
                kw = {"b": z} if which == "target" else {"s": z}
                assert st(**kw) == O.TREE_NONFINITE, (ver.__name__, bad, which)
        z = zb.copy()
        z[0, :] = -np.inf
        assert st(b=z) == O.TREE_NONFINITE
        z = zs.copy()
        z[0, 0] = -np.inf           # X1's token a cannot be drafted
        assert st(s=z) == O.TREE_NONFINITE
        # a leaf's draft row is never read
        z = zs.copy()
        z[3, :] = np.nan
        r = ver(par, tok, zb, z, T, u, W_)
        assert r.status == O.TREE_OK and r.accepted_node == base.accepted_node
    # Traversal Verification rejects X3 (a leaf) here: its target row is not read
    z = zb.copy()
    z[3, :] = np.nan
    r = O.verify_tree(par, tok, z, zs, T, u, W_)
    assert r.status == O.TREE_OK and r.accepted_node == 2
    # ... but it is read when X3 is accepted (Y ~ its target)
    r = O.verify_tree(par, tok, z, zs, T, np.zeros(6, np.float32), W_)
    assert r.status == O.TREE_NONFINITE


# ---------------------------------------------------------------------------
# LM head and row statistics (the inputs' normalisers)
# ---------------------------------------------------------------------------

def _bf16_bits(a):
    a = np.asarray(a, dtype=np.float32)
    return (a.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def pin_lmhead_logits():
    """The logits of bf16 inputs against a brute-force triple loop on a small
    case whose products and sums are exact (small integers and halves), the
    weight read as [vocab][hidden]; and every exact logit within the
    accumulation bound's own magnitude."""
    rng = np.random.default_rng(31)
    M, K, N = 5, 12, 7
    x = rng.integers(-4, 5, (M, K)) / 2.0
    w = rng.integers(-4, 5, (N, K)) / 2.0
    xb, wb = _bf16_bits(x), _bf16_bits(w)
    z = LM.logits(xb, wb)
    for m in range(M):
        for n in range(N):
            want = 0.0
            for k in range(K):
                want += float(x[m][k]) * float(w[n][k])
            assert z[m][n] == want, (m, n, z[m][n], want)
    bound = LM.accumulation_bound(xb, wb)
    assert np.all(np.abs(z) <= bound) and bound.shape == (M, N)


def pin_row_stats():
    """Row maximum and sum exp((z - max) / T) against scipy's logsumexp
    (log(sum) + max / T = logsumexp(z / T)), the softmax identity (the
    normalised terms sum to 1), the temperature's scaling, and the special
    rows: all -inf gives (-inf, 0), a NaN or +inf gives a non-finite sum."""
    from scipy.special import logsumexp
    rng = np.random.default_rng(32)
    z = rng.normal(0, 3, (6, 50))
    z[2, 7] = -np.inf
    for T in (0.2, 0.7, 1.0, 1.9):
        Tf = float(np.float32(T))
        m, s = LM.row_stats(z, T)
        assert np.array_equal(m, z.max(axis=1))
        np.testing.assert_allclose(np.log(s) + m / Tf, logsumexp(z / Tf, axis=1), rtol=0,
                                   atol=1e-12)
        p = np.exp((z - m[:, None]) / Tf) / s[:, None]
        np.testing.assert_allclose(p.sum(axis=1), 1.0, atol=1e-12)
    m, s = LM.row_stats(2.0 * z, 2.0)
    np.testing.assert_allclose(m, 2.0 * z.max(axis=1), atol=0)
    np.testing.assert_allclose(s, np.exp(z - z.max(axis=1, keepdims=True)).sum(axis=1),
                               rtol=1e-13)
    special = np.array([[-np.inf, -np.inf, -np.inf], [0.0, np.nan, 1.0], [0.0, np.inf, 1.0]])
    m, s = LM.row_stats(special, 1.0)
    assert m[0] == -np.inf and s[0] == 0.0
    assert not np.isfinite(s[1]) and not np.isfinite(s[2])
    # bf16 bit patterns are widened exactly first
    zb = _bf16_bits(z[:, :8])
    m2, _ = LM.row_stats(zb, 1.0)
    assert np.array_equal(m2, O.to_f64(zb).max(axis=1))


FAST_PINS = [pin_worked_example_trace, pin_worked_example_tokenlevel, pin_worked_example_law,
             pin_single_token_table1, pin_rrsw_example, pin_tempered_softmax_inverse,
             pin_inverse_cdf_law, pin_identical_models, pin_depth1_equals_rrsw,
             pin_invariants, pin_early_rejection_worked_example, pin_early_rejection_sound,
             pin_draft_sampler_law, pin_draft_sampler_statuses, pin_committed_sequence,
             pin_counters_worked_example, pin_counters_identical_models, pin_bf16_widening,
             pin_verifier_statuses, pin_lmhead_logits, pin_row_stats]
ENUM_PINS = [pin_lossless_exact, pin_lossless_irregular_T07, pin_chain_optimality]
ALL_PINS = FAST_PINS + ENUM_PINS


def first_failure(pins=ALL_PINS):
    """Name of the first pin that fails (or raises), or None."""
    for pin in pins:
        try:
            pin()
        except Exception:          # noqa: BLE001 - any failure counts
            return pin.__name__
    return None
