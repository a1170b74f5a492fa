"""Pins of the oracle's grouped-query score (a reading: K/V head h is scored
by the proxy rows of its q_group query heads; Section 5.1 F_score per query
head), independent of the oracle's own grouping loop."""

import math

import numpy as np
import pytest

from oracle import proxy_scores, proxy_scores_grouped


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def _brute_grouped(Q, K, pos, s, g):
    """Scalar loops: for every query head hq, its rows attend K/V head hq // g;
    each proxy row's causal softmax is added to that K/V head's column sums."""
    B, Hq, L, D = Q.shape
    H = K.shape[1]
    F = [[[0.0] * L for _ in range(H)] for _ in range(B)]
    for b in range(B):
        for hq in range(Hq):
            h = hq // g
            for p in pos:
                logits = [s * sum(float(Q[b, hq, p, d]) * float(K[b, h, j, d]) for d in range(D))
                          for j in range(p + 1)]
                mx = max(logits)
                den = sum(math.exp(x - mx) for x in logits)
                for j, x in enumerate(logits):
                    F[b][h][j] += math.exp(x - mx) / den
    return np.array(F)


def test_grouped_matches_brute_force():
    B, H, g, L, D = 2, 2, 3, 11, 4
    Q = _rand((B, H * g, L, D), 1)
    K = _rand((B, H, L, D), 2)
    pos = [3, 7, 10]
    F, _ = proxy_scores_grouped(Q, K, pos, 0.6, g)
    np.testing.assert_allclose(F, _brute_grouped(Q, K, pos, 0.6, g), rtol=1e-12, atol=1e-14)


def test_grouped_equals_multi_head_on_repeated_keys():
    """Grouped-query attention is multi-head attention whose K is repeated for
    the g query heads of a group (heads h*g .. h*g+g-1 read K/V head h): the
    grouped score of K/V head h is the sum of those g heads' scores."""
    B, H, g, L, D = 2, 3, 4, 40, 8
    Q = _rand((B, H * g, L, D), 3)
    K = _rand((B, H, L, D), 4)
    pos = list(range(30, 40))
    F, lse = proxy_scores_grouped(Q, K, pos, 0.35, g)
    Frep, lrep = proxy_scores(Q, np.repeat(K, g, axis=1), pos, 0.35)
    np.testing.assert_allclose(F, Frep.reshape(B, H, g, L).sum(axis=2), rtol=1e-12)
    np.testing.assert_allclose(lse, lrep, rtol=1e-12)


def test_grouped_mass_and_single_group():
    B, H, g, L, D = 1, 4, 2, 64, 16
    Q = _rand((B, H * g, L, D), 5)
    K = _rand((B, H, L, D), 6)
    pos = [5, 20, 40, 63]
    F, _ = proxy_scores_grouped(Q, K, pos, 0.25, g)
    np.testing.assert_allclose(F.sum(-1), len(pos) * g, rtol=1e-12)   # each row sums to 1
    F1, _ = proxy_scores_grouped(Q[:, ::g], K, pos, 0.25, 1)           # q_group = 1: multi-head
    Fm, _ = proxy_scores(Q[:, ::g], K, pos, 0.25)
    np.testing.assert_allclose(F1, Fm, rtol=1e-15)


def test_identical_query_heads_scale_the_score():
    """A group whose g query heads are identical scores g times one head."""
    B, H, g, L, D = 1, 2, 3, 30, 8
    q1 = _rand((B, H, L, D), 7)
    Q = np.repeat(q1, g, axis=1)
    K = _rand((B, H, L, D), 8)
    pos = [10, 29]
    F, _ = proxy_scores_grouped(Q, K, pos, 0.5, g)
    Fm, _ = proxy_scores(q1, K, pos, 0.5)
    np.testing.assert_allclose(F, g * Fm, rtol=1e-12)


def test_head_mapping_is_contiguous_groups():
    """Query head hq reads K/V head hq // g (contiguous groups), not hq % H:
    with K/V heads that differ, swapping to the strided mapping changes F."""
    B, H, g, L, D = 1, 2, 2, 20, 4
    Q = _rand((B, H * g, L, D), 9)
    K = _rand((B, H, L, D), 10)
    pos = [19]
    F, _ = proxy_scores_grouped(Q, K, pos, 1.0, g)
    strided = np.zeros_like(F)
    for hq in range(H * g):
        Fe, _ = proxy_scores(Q[:, hq:hq + 1], K[:, hq % H:hq % H + 1], pos, 1.0)
        strided[:, hq % H] += Fe[:, 0]
    assert not np.allclose(F, strided)
    np.testing.assert_allclose(F, _brute_grouped(Q, K, pos, 1.0, g), rtol=1e-12)
