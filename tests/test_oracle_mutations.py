"""Power of the oracle's pins: plant a plausible mistake in one step of the
oracle (on the CPU, via monkeypatch) and check that some pin fails."""

import numpy as np
import pytest

import oracle.tv_oracle as O
import oracle_pins as P


def _e1_without_p(p, b, s):
    d = np.maximum(b - s, 0.0)
    return d, float(d.sum())


def _e1_swapped(p, b, s):
    d = np.maximum(p * s - b, 0.0)
    return d, float(d.sum())


def _e2_no_renorm(s, x):
    s = s.copy()
    s[x] = 0.0
    return s


def _e2_wrong_token(s, x):
    s = s.copy()
    s[(x + 1) % len(s)] = 0.0
    return s / s.sum()


def _e2_always(s, x):
    return _e2_orig(s, x)


_e2_orig = O.draft_update_e2


def _e3_plus_p(S, p):
    return S / (S + p)


def _e3_no_missing_mass(S, p):
    return S / (S + 1.0)


def _rate_swapped(p, b, s, x):
    if p == 0.0 or s[x] == 0.0:
        return 0.0
    return min(p * s[x] / b[x], 1.0)


def _rate_no_clip(p, b, s, x):
    if p == 0.0 or b[x] == 0.0:
        return 0.0
    return p * b[x] / s[x]


def _no_rerate(*args):
    return None


def _softmax_no_temperature(z, T):
    return _softmax_orig(z, 1.0)


_softmax_orig = O.tempered_softmax


def _structure_reversed(parents, tokens, V, mode):
    st, children, depth = _structure_orig(parents, tokens, V, mode)
    if children is not None:
        children = [list(reversed(c)) for c in children]
    return st, children, depth


_structure_orig = O._structure


def _residual_without_norm(b, s):
    return np.maximum(b - s, 0.0)


def _early_when_below(res, children, alive, p, uniforms, j):
    if j == 0 or any(alive[c] for c in children[j]):
        return
    if float(uniforms[j]) < p[j]:       # comparison the wrong way round
        res.early_rejections += 1
        res.early_nodes.append(j)


def _early_any_child(res, children, alive, p, uniforms, j):
    if j != 0 and float(uniforms[j]) >= p[j]:   # ignores the children still left
        res.early_rejections += 1
        res.early_nodes.append(j)


def _finish_parents_only(res, children, depth, parents, uniforms):
    """Counts only the parents of tested nodes as consulted rows."""
    res = _finish_orig(res, children, depth, parents, uniforms)
    res.rows_consulted = len({int(parents[t]) for t in res.test_order})
    return res


def _finish_counts_accepted_row(res, children, depth, parents, uniforms):
    """Counts the accepted node's own row as consulted."""
    res = _finish_orig(res, children, depth, parents, uniforms)
    seen = set()
    for t in res.test_order:
        a = int(parents[t])
        while a >= 0:
            seen.add(a)
            a = int(parents[a])
    seen.add(res.accepted_node)
    res.rows_consulted = len(seen)
    return res


def _finish_tests_off_by_one(res, children, depth, parents, uniforms):
    res = _finish_orig(res, children, depth, parents, uniforms)
    res.tests = max(0, res.tests - 1)
    return res


def _finish_leaf_flag_inverted(res, children, depth, parents, uniforms):
    res = _finish_orig(res, children, depth, parents, uniforms)
    res.leaf_accepted = 1 - res.leaf_accepted
    return res


_finish_orig = O._finish


def _to_f64_as_fp16(logits):
    a = np.asarray(logits)
    if a.dtype == np.uint16:
        return a.view(np.float16).astype(np.float64)
    return a.astype(np.float64)


def _to_f64_low_half(logits):
    a = np.asarray(logits)
    if a.dtype == np.uint16:
        return a.astype(np.uint32).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def _structure_no_dup_check(parents, tokens, V, mode):
    return _structure_orig(parents, tokens, V, O.WITH_REPLACEMENT)


def _structure_token_bound_inclusive(parents, tokens, V, mode):
    return _structure_orig(parents, tokens, V + 1, mode)


MUTATIONS = {
    "e1 drops the p factor": ("residual_e1", _e1_without_p),
    "e1 target and draft swapped": ("residual_e1", _e1_swapped),
    "e2 does not renormalise": ("draft_update_e2", _e2_no_renorm),
    "e2 zeroes the wrong token": ("draft_update_e2", _e2_wrong_token),
    "e3 denominator S + p": ("acceptance_update_e3", _e3_plus_p),
    "e3 drops the missing mass": ("acceptance_update_e3", _e3_no_missing_mass),
    "chain rate ratio inverted": ("chain_rate", _rate_swapped),
    "chain rate not clipped at 1": ("chain_rate", _rate_no_clip),
    "no re-rating after an update": ("rerate_chains", _no_rerate),
    "temperature ignored": ("tempered_softmax", _softmax_no_temperature),
    "children visited last-first": ("_structure", _structure_reversed),
    "RRS residual not normalised": ("rrs_residual", _residual_without_norm),
    "early rejection with u below p": ("_early_rejection", _early_when_below),
    "early rejection with children left": ("_early_rejection", _early_any_child),
    "consulted rows: parents of tested nodes only": ("_finish", _finish_parents_only),
    "consulted rows include the accepted node": ("_finish", _finish_counts_accepted_row),
    "tests counter one short": ("_finish", _finish_tests_off_by_one),
    "leaf-accepted flag inverted": ("_finish", _finish_leaf_flag_inverted),
    "bf16 read as fp16": ("to_f64", _to_f64_as_fp16),
    "bf16 widened into the low half": ("to_f64", _to_f64_low_half),
    "duplicate siblings not detected": ("_structure", _structure_no_dup_check),
    "token bound V accepted": ("_structure", _structure_token_bound_inclusive),
}


def test_unmutated_oracle_passes_every_pin():
    assert P.first_failure() is None


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(monkeypatch, name):
    attr, fn = MUTATIONS[name]
    monkeypatch.setattr(O, attr, fn)
    assert P.first_failure() is not None, f"no pin catches: {name}"


def test_mismatched_sibling_pairing_is_not_lossless(monkeypatch):
    """Negative control for the sibling-mode reading: children drawn i.i.d. but
    verified with Eq. (e2) (duplicates allowed through) must break losslessness,
    while the matched pairings pass (pin_lossless_exact)."""
    import oracle.enumerate as E
    import workloads as W
    monkeypatch.setattr(O, "_structure",
                        lambda p, t, V, mode: _structure_orig(p, t, V, O.WITH_REPLACEMENT))
    m = W.ContextModel(3, seed=0)
    par = W.binary_parents(2)
    law = E.draft_tree_law(O.verify_tree, par, m, 1.0, O.WITH_REPLACEMENT,
                           O.WITHOUT_REPLACEMENT)
    assert E.law_distance(law, E.target_law(m, 1.0, 3)) > 1e-4


def test_two_leaf_sibling_counterexample(monkeypatch):
    """Root with two leaf children drawn i.i.d. from q = [.6,.3,.1], target
    [.3,.4,.3] (the Table 1 pair): the first-token law is the target with the
    matched update and [3/10, 17/50, 9/25] when Eq. (e2) zeroes a duplicate."""
    import oracle.enumerate as E

    class M:
        vocab = 3

        def target(self, ctx):
            return np.log([.3, .4, .3])

        def draft(self, ctx):
            return np.log([.6, .3, .1])

    par = np.array([-1, 0, 0], np.int32)

    def first_token(law):
        out = np.zeros(3)
        for seq, pr in law.items():
            out[seq[0]] += pr
        return out

    good = first_token(E.draft_tree_law(O.verify_tree, par, M(), 1.0, O.WITH_REPLACEMENT,
                                        O.WITH_REPLACEMENT, length=1))
    np.testing.assert_allclose(good, [.3, .4, .3], atol=1e-12)
    monkeypatch.setattr(O, "_structure",
                        lambda p, t, V, mode: _structure_orig(p, t, V, O.WITH_REPLACEMENT))
    bad = first_token(E.draft_tree_law(O.verify_tree, par, M(), 1.0, O.WITH_REPLACEMENT,
                                       O.WITHOUT_REPLACEMENT, length=1))
    np.testing.assert_allclose(bad, [3 / 10, 17 / 50, 9 / 25], atol=1e-12)


def _sampler_with_replacement(parents, draft_logits, temperature, uniforms, mode=0):
    import oracle.draft_sampler as DS
    return _draw_orig(parents, draft_logits, temperature, uniforms, O.WITH_REPLACEMENT)


def _sampler_no_temperature(parents, draft_logits, temperature, uniforms, mode=0):
    return _draw_orig(parents, draft_logits, 1.0, uniforms, mode)


import oracle.draft_sampler as _DS  # noqa: E402

_draw_orig = _DS.draw_tree_tokens


@pytest.mark.parametrize("fn", [_sampler_with_replacement, _sampler_no_temperature])
def test_sampler_mutation_is_caught(monkeypatch, fn):
    """The sampler pins catch siblings drawn with replacement where they must
    not repeat, and an ignored temperature."""
    monkeypatch.setattr(_DS, "draw_tree_tokens", fn)
    assert P.first_failure([P.pin_draft_sampler_law, P.pin_draft_sampler_statuses]) is not None


import oracle.lmhead as _LM  # noqa: E402

_lm_logits_orig = _LM.logits
_lm_stats_orig = _LM.row_stats


def _lm_logits_dropped_last_k(hidden, weight):
    x = O.to_f64(hidden)[:, :-1]
    w = O.to_f64(weight)[:, :-1]
    return x @ w.T


def _lm_stats_no_temperature(z, T):
    return _lm_stats_orig(z, 1.0)


def _lm_stats_unshifted(z, T):
    z = O.to_f64(z)
    T = float(np.float32(T))
    return z.max(axis=-1), np.exp(z / T).sum(axis=-1)


@pytest.mark.parametrize("attr,fn", [("logits", _lm_logits_dropped_last_k),
                                     ("row_stats", _lm_stats_no_temperature),
                                     ("row_stats", _lm_stats_unshifted)])
def test_lmhead_mutation_is_caught(monkeypatch, attr, fn):
    """The LM-head pins catch a dropped hidden column, an ignored temperature
    and a sum taken without the maximum subtracted."""
    monkeypatch.setattr(_LM, attr, fn)
    assert P.first_failure([P.pin_lmhead_logits, P.pin_row_stats]) is not None
