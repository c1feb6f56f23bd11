"""The four-scalar form of a node's state that the HIP kernels use, checked on
the CPU against the oracle's literal vector updates.

After k rejections at a node with original target p, draft q and starting rate
pi_0, Algorithm 3 holds vectors b_k, s_k. The kernels keep only (pi, A, B, c):
b_k = [A p - B q]_+, s_k = c q off the rejected tokens (c = 1/(1 - q(rejected))
without replacement, 1 with), and per rejection
  S = sum [alpha p - beta q]_+,  alpha = pi A,  beta = pi B + c,
  A <- alpha / S,  B <- beta / S,  pi <- S / (S + (1 - pi)),
so a sibling's ratio is b/s = [A r - B]_+ / c with r = p / q. This holds because
a rejected token always had pi b(x) < s(x) (a chain rate of 1 cannot be
rejected), so clipping commutes with the linear update."""

import numpy as np
import pytest

import oracle.tv_oracle as O


@pytest.mark.parametrize("mode", [O.WITHOUT_REPLACEMENT, O.WITH_REPLACEMENT])
def test_four_scalar_state_matches_literal_vectors(mode):
    rng = np.random.default_rng(2024 + mode)
    worst = 0.0
    for case in range(2000):
        V = 50
        p = O.tempered_softmax(rng.normal(0, 2, V), 1.0)
        q = O.tempered_softmax(np.log(p) + rng.normal(0, 1, V), 1.0)
        pi = 1.0 if case % 4 == 0 else float(rng.uniform(0.05, 1.0))
        b, s = p.copy(), q.copy()
        A, Bc, zmass = 1.0, 0.0, 0.0
        rejected = []
        for step in range(6):
            c = 1.0 / (1.0 - zmass)
            ratio_lit = np.divide(b, s, out=np.zeros(V), where=s > 0)
            ratio_cf = np.maximum(A * (p / q) - Bc, 0.0) / c
            live = [x for x in range(V) if x not in rejected]
            worst = max(worst, float(np.max(np.abs(ratio_lit[live] - ratio_cf[live])
                                            / np.maximum(1.0, ratio_lit[live]))))
            # a token that can be rejected: chain rate pi * b/s below 1
            cand = [x for x in live if pi * ratio_lit[x] < 1.0 and q[x] > 0]
            if not cand or pi == 0.0:
                break
            x = int(rng.choice(cand))
            # literal Eq. (e1)-(e3)
            d, S = O.residual_e1(pi, b, s)
            alpha, beta = pi * A, pi * Bc + c
            S_cf = float(np.maximum(alpha * p - beta * q, 0.0).sum())
            worst = max(worst, abs(S - S_cf) / max(S, 1e-300) if S > 0 else abs(S_cf))
            if S <= 0.0:
                break
            b = d / S
            if mode == O.WITHOUT_REPLACEMENT:
                s = O.draft_update_e2(s, x)
                zmass += q[x]
                rejected.append(x)
            pi = O.acceptance_update_e3(S, pi)
            A, Bc = alpha / S, beta / S
            np.testing.assert_allclose(b, np.maximum(A * p - Bc * q, 0.0), atol=1e-12)
            if mode == O.WITHOUT_REPLACEMENT:
                cnew = 1.0 / (1.0 - zmass)
                mask = np.ones(V, bool)
                mask[rejected] = False
                np.testing.assert_allclose(s[mask], cnew * q[mask], rtol=1e-10)
                assert np.all(s[~mask] == 0.0)
            else:
                np.testing.assert_allclose(s, q, rtol=0, atol=0)
    assert worst < 1e-9, worst
