"""The GPU-vs-oracle keep-set rule itself (tests/_parity.py) on the CPU: near
ties at either selection boundary pass, any other difference fails.  The
"GPU" sets here are the oracle's own sets with planted changes."""

import numpy as np
import pytest

from oracle import SAMPLE_SOFTMAX, select_head
from tests._parity import check_keep_near, check_scores


def _head(L=3000, P=16, C=600, Cr=300, seed=3):
    rng = np.random.default_rng(seed)
    F = rng.gamma(0.4, 1.0, size=L).astype(np.float32)
    pos = list(range(L - P, L))
    ref = select_head(F, pos, P, C, Cr, SAMPLE_SOFTMAX, 1, 0, 0, 0)
    return F, pos, ref


def _swap(keep, out_tok, in_tok):
    s = set(keep.tolist())
    s.remove(out_tok)
    s.add(in_tok)
    return np.array(sorted(s))


def test_identical_sets_pass():
    F, pos, ref = _head()
    assert check_keep_near(ref["keep"], ref, F, 300) == 0


def test_far_swap_fails():
    """Dropping the best-scored token for the worst candidate is no near tie."""
    F, pos, ref = _head()
    us = ref["u_score"]
    best = int(us[np.argmax(F[us])])
    outside = sorted(set(range(len(F) - 16)) - set(ref["keep"].tolist()))
    worst = min(outside, key=lambda j: F[j])
    with pytest.raises(AssertionError, match="not a near-tie"):
        check_keep_near(_swap(ref["keep"], best, worst), ref, F, 300)


def test_score_boundary_near_tie_passes():
    """Two tokens whose scores differ by far less than 1e-3 relative, one
    just inside u_score, one just outside: a swap is allowed."""
    F, pos, ref = _head()
    us = ref["u_score"]
    t = int(us[np.argmin(F[us])])             # the Cp-th best
    F = F.copy()
    cand = [j for j in range(len(F) - 16) if j not in set(ref["keep"].tolist())]
    j = min(cand, key=lambda x: ref["key"][x])   # the candidate least likely to be drawn
    F[j] = np.float32(F[t] * (1 - 2e-4))      # a near tie just below the boundary
    ref = select_head(F, pos, 16, 600, 300, SAMPLE_SOFTMAX, 1, 0, 0, 0)
    if j in ref["keep"]:
        pytest.skip("the planted token was drawn at random")
    assert check_keep_near(_swap(ref["keep"], t, j), ref, F, 300) == 2


def test_random_boundary_without_a_tie_fails():
    """Swapping the last random pick for the next one in key order is a
    difference only a key near-tie (or a score-boundary cascade) explains;
    with a clear key gap and no score tie band, it fails.  Scores are
    geometric (0.5 % apart), so no two lie within 1e-3 of each other."""
    L, P = 1000, 16
    rng = np.random.default_rng(8)
    F = (1e-3 * 1.005 ** rng.permutation(L)).astype(np.float32)
    pos = list(range(L - P, L))
    ref = select_head(F, pos, P, 600, 300, SAMPLE_SOFTMAX, 1, 0, 0, 0)
    key = ref["key"].astype(np.float64)
    R2 = np.array(sorted(set(range(len(F) - 16)) - set(ref["u_score"].tolist())))
    order = R2[np.lexsort((R2, -key[R2]))]
    last, nxt = int(order[299]), int(order[300])
    gap = key[last] - key[nxt]
    us = ref["u_score"]
    T1 = F[us].min()
    band = np.abs(F[R2] - T1) <= 1e-3 * T1
    if gap <= 1e-3 * (F[last] + F[nxt]) + 1e-6 or band.any():
        pytest.skip("seed gives a near tie at the boundary")
    with pytest.raises(AssertionError, match="not a near-tie"):
        check_keep_near(_swap(ref["keep"], last, nxt), ref, F, 300)


def test_score_floor_is_1e30():
    """Scores at or above 1e-30 must match to 1e-3 relative; flushing one of
    them to zero fails, flushing a value below the floor passes."""
    ref = np.array([0.5, 2e-30, 1e-31])
    check_scores(np.array([0.5, 2e-30, 0.0]), ref)
    with pytest.raises(AssertionError):
        check_scores(np.array([0.5, 0.0, 0.0]), ref)
