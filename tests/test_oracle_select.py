"""Pins of the oracle's keep-set selection (Section 5.1 argmax, Section 5.2
random eviction, Algorithm 1 union) and compaction (Section 3)."""

import json
import os
from collections import Counter
from fractions import Fraction
import math

import numpy as np
import pytest
import scipy.stats

from oracle import (SAMPLE_PROPORTIONAL, SAMPLE_SOFTMAX, SAMPLE_UNIFORM,
                    budget_split, compact, protected_set, select, select_head,
                    top_k_lower_index)
from oracle.sampling import sequential_sample, set_probabilities

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_numbers.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def test_topk_brute_force_with_ties():
    rng = np.random.default_rng(0)
    for trial in range(50):
        L = int(rng.integers(1, 40))
        vals = rng.integers(0, 5, size=L).astype(np.float32)  # many ties
        cand = np.sort(rng.choice(L, size=int(rng.integers(0, L + 1)), replace=False))
        k = int(rng.integers(0, len(cand) + 1))
        got = top_k_lower_index(vals, cand, k)
        ref = sorted(cand.tolist(), key=lambda j: (-float(vals[j]), j))[:k]
        assert got.tolist() == ref


def _check_keep(keep, L, C, Pi):
    assert keep.shape == (C,)
    assert (np.diff(keep) > 0).all(), "strictly ascending"
    assert keep.min(initial=0) >= 0 and keep.max(initial=0) < max(L, 1)
    assert set(Pi.tolist()) <= set(keep.tolist())


@pytest.mark.parametrize("mode", [SAMPLE_SOFTMAX, SAMPLE_PROPORTIONAL, SAMPLE_UNIFORM])
def test_keep_set_structure(mode):
    rng = np.random.default_rng(1)
    L, P = 500, 20
    pos = list(range(L - P, L))
    F = rng.gamma(0.5, 1.0, size=L).astype(np.float32)
    for n_protect, C, Cr in [(P, 100, 60), (P, P, 0), (0, 100, 100), (5, 500, 0),
                             (P, 500, 480), (10, 10, 0), (0, 0, 0)]:
        r = select_head(F, pos, n_protect, C, Cr, mode, 7, 3, 0, 1)
        _check_keep(r["keep"], L, C, r["protected"])
        Cp = C - n_protect - Cr
        assert len(r["u_score"]) == Cp and len(r["u_random"]) == Cr
        parts = np.concatenate([r["protected"], r["u_score"], r["u_random"]])
        assert len(np.unique(parts)) == C, "the three parts are disjoint"
        # top-Cp dominates every other candidate of R
        R = np.setdiff1d(np.arange(L), r["protected"])
        rest = np.setdiff1d(R, r["u_score"])
        if Cp and len(rest):
            assert F[r["u_score"]].min() >= F[rest].max()


def test_budget_reading_matches_hyperparameter_table():
    """Appendix A.6: Protect + Proxy-Tokens Eviction + Random = Budget in every
    row, so protected proxies count inside C."""
    for row in _golden()["budget_table"]["rows"]:
        L = 2000  # tokens; every column is a whole number of tokens at this L
        C = round(row["budget"] * L / 100)
        n_protect = round(row["protect"] * L / 100)
        Cr = round(row["random"] * L / 100)
        assert budget_split(C, Cr, n_protect) == round(row["proxy_evict"] * L / 100)


def test_kv_cache_size_of_headline_workload():
    """Section 1: 7B model (32 layers, hidden 4096), batch 4, 32k -> 64GB."""
    from synth import WORKLOADS
    g = _golden()["kv_cache_size"]
    w = WORKLOADS["prefill_32k"]
    assert (w.layers, w.H * w.D, w.B, w.L) == (g["layers"], g["hidden"], g["batch"], g["seq"])
    total = 2 * w.layers * w.B * w.L * w.H * w.D * g["bytes_per_elt"]
    assert total == g["printed_gb"] * 2 ** 30


def _empirical_sets(weights_F, mode, k, n_seeds):
    L = len(weights_F)
    cnt = Counter()
    for seed in range(n_seeds):
        r = select_head(weights_F, [L - 1], 0, k, k, mode, seed, 0, 0, 0)
        cnt[tuple(r["u_random"].tolist())] += 1
    return cnt


@pytest.mark.parametrize("mode", [SAMPLE_SOFTMAX, SAMPLE_PROPORTIONAL, SAMPLE_UNIFORM])
def test_sampling_law_is_successive_draws(mode):
    """Gumbel-top-k on the oracle's keys reproduces the exact Plackett-Luce law
    of drawing Cr tokens one by one from the normalised distribution
    (Section 5.2), checked by a chi-square test over many seeds."""
    F = np.array([0.1, 1.3, 0.02, 2.2, 0.7, 0.45], dtype=np.float32)
    if mode == SAMPLE_SOFTMAX:
        w = np.exp(F.astype(np.float64))
    elif mode == SAMPLE_PROPORTIONAL:
        w = F.astype(np.float64)
    else:
        w = np.ones_like(F, dtype=np.float64)
    k, n = 3, 6000
    exact = set_probabilities(w, k)
    emp = _empirical_sets(F, mode, k, n)
    keys = sorted(exact)
    obs = np.array([emp.get(s, 0) for s in keys], dtype=np.float64)
    exp = np.array([exact[s] * n for s in keys])
    assert abs(obs.sum() - n) < 1e-9
    stat, p = scipy.stats.chisquare(obs, exp)
    assert p > 1e-3, (stat, p)


def test_sequential_sampler_agrees_with_exact_law():
    """The literal one-at-a-time sampler itself follows the exact law (this
    pins the helper used above)."""
    w = np.array([0.5, 2.0, 1.0, 0.25, 3.0])
    k, n = 2, 8000
    exact = set_probabilities(w, k)
    rng = np.random.default_rng(3)
    emp = Counter(sequential_sample(w, k, rng) for _ in range(n))
    keys = sorted(exact)
    stat, p = scipy.stats.chisquare([emp.get(s, 0) for s in keys], [exact[s] * n for s in keys])
    assert p > 1e-3


def test_uniform_inclusion_is_hypergeometric():
    """UNIFORM keeps each remaining candidate with probability Cr / |R2|."""
    L, C, Cr, P = 64, 24, 16, 4
    pos = list(range(L - P, L))
    F = np.linspace(0.01, 1, L).astype(np.float32)
    hits = np.zeros(L)
    n = 1500
    for seed in range(n):
        hits[select_head(F, pos, P, C, Cr, SAMPLE_UNIFORM, seed, 0, 0, 0)["u_random"]] += 1
    Cp = C - P - Cr
    R2 = np.arange(L - P - Cp)  # top-Cp takes the largest F, i.e. the highest indices of R
    rate = hits[R2] / n
    p_in = Cr / len(R2)
    sd = math.sqrt(p_in * (1 - p_in) / n)
    assert abs(rate.mean() - p_in) < 3 * sd / math.sqrt(len(R2)) + 1e-9
    assert np.abs(rate - p_in).max() < 5 * sd
    assert hits[L - P - Cp:].sum() == 0


def test_headwise_retention_matches_paper():
    """Section 6.4: with independent per-head draws at C = 20 %, a token
    survives in at least one of 32 heads with probability 99.92 %."""
    g = _golden()["headwise_retention"]
    H, L = g["heads"], 4096
    C = int(g["budget"] * L)
    F = np.full((1, H, L), 1.0 / L, dtype=np.float32)
    keep = select(F, [L - 1], 0, C, C, SAMPLE_UNIFORM, 11, 0)
    kept_any = np.zeros(L, dtype=bool)
    for h in range(H):
        kept_any[keep[0, h]] = True
    frac = kept_any.mean() * 100
    theory = (1 - (1 - g["budget"]) ** H) * 100
    assert round(theory, 2) == g["printed_percent"]
    assert abs(frac - g["printed_percent"]) < 0.15


def test_layerwise_retention_bound():
    """Section 6.4: at C = 1 %, across 32 layers x 32 heads, retention exceeds
    99.99 %.  Each (layer, head) draws its own Philox stream."""
    g = _golden()["layerwise_retention"]
    H, layers, L = g["heads"], g["layers"], 2048
    C = max(1, int(g["budget"] * L))
    F = np.full((1, H, L), 1.0 / L, dtype=np.float32)
    kept_any = np.zeros(L, dtype=bool)
    for layer in range(layers):
        keep = select(F, [L - 1], 0, C, C, SAMPLE_UNIFORM, 5, layer)
        for h in range(H):
            kept_any[keep[0, h]] = True
    assert kept_any.mean() * 100 > g["printed_lower_bound_percent"] - 0.1
    assert (1 - (1 - C / L) ** (H * layers)) * 100 > g["printed_lower_bound_percent"]


def test_streams_differ_per_head_and_layer_and_repeat_per_seed():
    L = 1000
    F = np.random.default_rng(4).random((2, 2, L)).astype(np.float32)
    a = select(F, [L - 1], 1, 200, 150, SAMPLE_SOFTMAX, 9, 0)
    b = select(F, [L - 1], 1, 200, 150, SAMPLE_SOFTMAX, 9, 0)
    c = select(F, [L - 1], 1, 200, 150, SAMPLE_SOFTMAX, 9, 1)
    d = select(F, [L - 1], 1, 200, 150, SAMPLE_SOFTMAX, 10, 0)
    assert np.array_equal(a, b)
    assert not np.array_equal(a, c) and not np.array_equal(a, d)
    F2 = np.broadcast_to(F[:1, :1], F.shape).copy()
    e = select(F2, [L - 1], 1, 200, 150, SAMPLE_SOFTMAX, 9, 0)
    assert not np.array_equal(e[0, 0], e[0, 1]) and not np.array_equal(e[0, 0], e[1, 0])


def test_compact_is_exact_row_copy():
    rng = np.random.default_rng(5)
    B, H, L, D, C = 2, 3, 50, 8, 12
    K = rng.standard_normal((B, H, L, D)).astype(np.float32)
    V = rng.standard_normal((B, H, L, D)).astype(np.float32)
    idx = np.sort(np.stack([[rng.choice(L, C, replace=False) for _ in range(H)] for _ in range(B)]), -1)
    Kc, Vc = compact(K, V, idx)
    for b in range(B):
        for h in range(H):
            for c in range(C):
                assert Kc[b, h, c].tobytes() == K[b, h, idx[b, h, c]].tobytes()
                assert Vc[b, h, c].tobytes() == V[b, h, idx[b, h, c]].tobytes()
    assert Kc.nbytes == B * H * C * D * 4


def test_protected_set_is_the_last_proxies():
    """Reading of "Protect Proxy" (Appendix A.6) with Section 5.1's default
    (proxies are kept): the force-kept set is the last n_protect proxies in
    position order, none for n_protect = 0, all of them for n_protect = P.
    Expected sets are written out, not computed by slicing."""
    pos = [3, 8, 20, 41, 77]
    expected = {0: [], 1: [77], 2: [41, 77], 4: [8, 20, 41, 77], 5: [3, 8, 20, 41, 77]}
    for n, want in expected.items():
        assert protected_set(pos, n).tolist() == want, n
    for bad in (-1, 6):
        with pytest.raises(ValueError):
            protected_set(pos, bad)


def test_unprotected_proxy_competes_in_R():
    """With n_protect < P the first P - n_protect proxies are ordinary
    candidates of R (Section 5.1 argmax over R): an unprotected proxy with the
    largest score is taken by u_score, one with a tiny score is not kept, and
    a protected proxy with score 0 is kept anyway."""
    L, C, Cr = 40, 8, 0
    pos = [30, 31, 32, 33]                # proxies; the last two are protected
    F = np.full(L, 0.01, dtype=np.float32)
    F[30] = 5.0                           # unprotected proxy, top score
    F[31] = 1e-6                          # unprotected proxy, bottom score
    F[32] = 0.0                           # protected proxy, score 0
    F[[2, 9, 17, 25, 38]] = [0.5, 0.4, 0.3, 0.2, 0.1]
    r = select_head(F, pos, 2, C, Cr, SAMPLE_SOFTMAX, 0, 0, 0, 0)
    assert r["protected"].tolist() == [32, 33]
    assert r["u_score"].tolist() == [2, 9, 17, 25, 30, 38]
    assert r["keep"].tolist() == [2, 9, 17, 25, 30, 32, 33, 38]
    assert 31 not in r["keep"]
