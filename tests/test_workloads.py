"""The seeded input generators (no GPU): tree shapes are valid and have the
sizes and depths their workloads state."""

import numpy as np

import workloads as W


def _valid(parents):
    return parents[0] == -1 and all(0 <= parents[i] < i for i in range(1, len(parents)))


def test_irregular_trees_have_exact_size_and_depth():
    rng = np.random.default_rng(0)
    for n, depth in ((60, 6), (64, 7)):
        for _ in range(5):
            p = W.geometric_bfs_parents(rng, n, depth)
            assert len(p) == n + 1 and _valid(p)
            assert W.node_depths(p).max() == depth
            assert np.bincount(p[1:]).max() <= 4          # branching 1..4


def test_deep_trees_reach_sequoia_scale():
    """767 draft nodes, parents within the 64 nodes before: depth above 20 and
    hundreds of nodes with children."""
    for b in range(4):
        p = W.windowed_parents(np.random.default_rng(b), 767, 64)
        assert len(p) == 768 and _valid(p)
        assert all(p[i] >= i - 64 for i in range(1, 768))
        assert W.node_depths(p).max() > 20
        assert len(set(p[1:].tolist())) > 300


def test_uniforms_are_exact_in_float32():
    u = W.uniforms_np(np.random.default_rng(1), (64, 65))
    assert u.dtype == np.float32 and (u >= 0).all() and (u < 1).all()
    k = u.astype(np.float64) * 2.0 ** 24
    assert np.array_equal(k, np.round(k))                # multiples of 2^-24
