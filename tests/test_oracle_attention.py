"""Pins of the oracle's causal attention and per-row log-sum-exp (the forward
pass whose log-sum-exp Appendix A.7 feeds to the score), each against
something other than the oracle's own formula: scalar loops, torch's and
scipy's library routines, closed forms and limits."""

import math

import numpy as np
import pytest
import torch
from scipy.special import logsumexp

from oracle import causal_attention, proxy_scores_grouped


def _rand(shape, seed, scale=1.0):
    return scale * np.random.default_rng(seed).standard_normal(shape)


def _brute(Q, K, V, s, g):
    """Scalar loops over (b, hq, i): softmax over keys j <= i of K/V head
    hq // g, then the weighted sum of V rows."""
    B, Hq, L, D = Q.shape
    O = np.zeros(Q.shape)
    lse = np.zeros((B, Hq, L))
    for b in range(B):
        for hq in range(Hq):
            h = hq // g
            for i in range(L):
                logits = [s * sum(float(Q[b, hq, i, d]) * float(K[b, h, j, d]) for d in range(D))
                          for j in range(i + 1)]
                mx = max(logits)
                den = sum(math.exp(x - mx) for x in logits)
                lse[b, hq, i] = mx + math.log(den)
                for j, x in enumerate(logits):
                    w = math.exp(x - mx) / den
                    for d in range(D):
                        O[b, hq, i, d] += w * float(V[b, h, j, d])
    return O, lse


@pytest.mark.parametrize("g", [1, 2])
def test_attention_matches_brute_force(g):
    B, H, L, D = 2, 2, 9, 5
    Q = _rand((B, H * g, L, D), 1)
    K = _rand((B, H, L, D), 2)
    V = _rand((B, H, L, D), 3)
    O, lse = causal_attention(Q, K, V, 0.7, q_group=g)
    Ob, lb = _brute(Q, K, V, 0.7, g)
    np.testing.assert_allclose(O, Ob, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, lb, rtol=1e-12, atol=1e-12)


def test_output_matches_torch_sdpa():
    B, H, L, D = 2, 3, 40, 16
    Q = _rand((B, H, L, D), 4)
    K = _rand((B, H, L, D), 5)
    V = _rand((B, H, L, D), 6)
    s = 1.0 / math.sqrt(D)
    O, _ = causal_attention(Q, K, V, s)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(Q), torch.from_numpy(K), torch.from_numpy(V), is_causal=True, scale=s)
    np.testing.assert_allclose(O, ref.numpy(), rtol=1e-12, atol=1e-12)


def test_lse_matches_scipy_logsumexp():
    B, H, L, D = 1, 2, 33, 8
    Q = _rand((B, H, L, D), 7, 2.0)
    K = _rand((B, H, L, D), 8, 2.0)
    V = _rand((B, H, L, D), 9)
    s = 0.35
    _, lse = causal_attention(Q, K, V, s)
    for h in range(H):
        for i in range(L):
            a = s * (Q[0, h, i] @ K[0, h, : i + 1].T)
            assert lse[0, h, i] == pytest.approx(logsumexp(a), rel=1e-13, abs=1e-13)


def test_zero_keys_average_the_prefix():
    """K = 0: every visible key has logit 0, so row i is the mean of V[0..i]
    and its log-sum-exp is log(i + 1)."""
    B, H, L, D = 1, 2, 17, 6
    Q = _rand((B, H, L, D), 10)
    K = np.zeros((B, H, L, D))
    V = _rand((B, H, L, D), 11)
    O, lse = causal_attention(Q, K, V, 0.9)
    for i in range(L):
        np.testing.assert_allclose(O[0, :, i], V[0, :, : i + 1].mean(axis=1), rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(lse[0, :, i], math.log(i + 1), rtol=0, atol=1e-13)


def test_hard_attention_limit_returns_own_value():
    """Orthogonal one-hot keys and queries with a large scale: row i's mass
    sits on key i, so O[i] -> V[i] and lse[i] -> s."""
    L = D = 12
    eye = np.eye(L)[None, None]
    V = _rand((1, 1, L, D), 12)
    O, lse = causal_attention(eye, eye, V, 60.0)
    np.testing.assert_allclose(O[0, 0], V[0, 0], rtol=0, atol=1e-20)
    np.testing.assert_allclose(lse[0, 0], 60.0, rtol=0, atol=1e-20)


def test_grouping_maps_query_head_to_kv_head_quotient():
    """Query head hq reads K/V head hq // g: the same as multi-head attention
    over K and V with each head repeated g times (and not hq mod H)."""
    B, H, g, L, D = 1, 3, 2, 10, 4
    Q = _rand((B, H * g, L, D), 13)
    K = _rand((B, H, L, D), 14)
    V = _rand((B, H, L, D), 15)
    O, lse = causal_attention(Q, K, V, 0.5, q_group=g)
    O1, l1 = causal_attention(Q, np.repeat(K, g, axis=1), np.repeat(V, g, axis=1), 0.5)
    np.testing.assert_allclose(O, O1, rtol=0, atol=0)
    np.testing.assert_allclose(lse, l1, rtol=0, atol=0)


def test_row_subset_and_proxy_rows():
    """Rows computed alone equal the same rows of the full computation, and at
    the proxy rows the log-sum-exp is the one the score's own pass 1 reaches
    (Algorithm 2 takes it from the attention instead)."""
    B, H, g, L, D = 2, 2, 2, 30, 8
    Q = _rand((B, H * g, L, D), 16)
    K = _rand((B, H, L, D), 17)
    V = _rand((B, H, L, D), 18)
    rows = np.array([0, 5, 17, 29])
    O, lse = causal_attention(Q, K, V, 0.4, q_group=g)
    Or, lr = causal_attention(Q, K, V, 0.4, q_group=g, rows=rows)
    np.testing.assert_allclose(Or, O[:, :, rows], rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(lr, lse[:, :, rows], rtol=1e-14, atol=1e-15)
    _, lse_p = proxy_scores_grouped(Q, K, rows, 0.4, g)
    np.testing.assert_allclose(lse_p, lse[:, :, rows], rtol=1e-13, atol=1e-13)
