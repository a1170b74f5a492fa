"""Pins of the oracle's proxy-token score (Section 5.1, F_score) against facts
the paper and the mathematics fix, independent of the oracle's own code."""

import math

import numpy as np
import pytest
import scipy.special
import torch

from oracle import proxy_scores

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def _brute(Q, K, pos, s):
    """Scalar loops with math.exp: softmax of each proxy row over its visible
    keys, summed per key."""
    B, H, L, D = K.shape
    F = [[[0.0] * L for _ in range(H)] for _ in range(B)]
    for b in range(B):
        for h in range(H):
            for p in pos:
                logits = []
                for j in range(p + 1):
                    dot = 0.0
                    for d in range(D):
                        dot += float(Q[b, h, p, d]) * float(K[b, h, j, d])
                    logits.append(s * dot)
                mx = max(logits)
                den = sum(math.exp(a - mx) for a in logits)
                for j, a in enumerate(logits):
                    F[b][h][j] += math.exp(a - mx) / den
    return np.array(F)


@pytest.mark.parametrize("L,D,pos,seed", [
    (7, 3, [6], 0), (12, 4, [3, 7, 11], 1), (16, 8, [0, 5, 6, 15], 2), (9, 2, [8], 3),
])
def test_brute_force_tiny(L, D, pos, seed):
    Q = _rand((2, 2, L, D), seed)
    K = _rand((2, 2, L, D), seed + 100)
    F, _ = proxy_scores(Q, K, pos, 0.7)
    np.testing.assert_allclose(F, _brute(Q, K, pos, 0.7), rtol=1e-12, atol=1e-14)


def test_row_mass_invariant():
    """Each proxy row is a probability distribution, so the head's total score
    mass equals the proxy count, every F lies in [0, P], and keys after the
    last proxy get nothing."""
    L, D = 300, 16
    pos = [40, 41, 100, 250, 251, 260]
    Q = _rand((2, 3, L, D), 5)
    K = _rand((2, 3, L, D), 6)
    F, _ = proxy_scores(Q, K, pos, 1 / 4)
    np.testing.assert_allclose(F.sum(-1), len(pos), rtol=1e-12)
    assert (F >= 0).all() and (F <= len(pos) + 1e-12).all()
    assert (F[..., pos[-1] + 1:] == 0).all()


def test_single_proxy_is_softmax_of_current_token():
    """With one proxy at the last position the score is the current token's
    attention distribution (the MSRNN special case, Section 5.1)."""
    L, D = 64, 8
    Q = _rand((1, 2, L, D), 7)
    K = _rand((1, 2, L, D), 8)
    for p in (L - 1, 37):
        F, _ = proxy_scores(Q, K, [p], 0.35)
        logits = 0.35 * torch.einsum("bhd,bhjd->bhj", torch.from_numpy(Q[:, :, p]),
                                     torch.from_numpy(K[:, :, : p + 1]))
        ref = torch.softmax(logits, dim=-1).numpy()
        np.testing.assert_allclose(F[..., : p + 1], ref, rtol=1e-12, atol=1e-15)
        assert (F[..., p + 1:] == 0).all()


def test_all_tokens_as_proxies_is_accumulated_attention():
    """With every token a proxy the score is the column sum of the full causal
    attention matrix (the H2O special case, Section 5.1)."""
    L, D = 48, 8
    Q = _rand((1, 2, L, D), 9)
    K = _rand((1, 2, L, D), 10)
    F, _ = proxy_scores(Q, K, list(range(L)), 0.3)
    q, k = torch.from_numpy(Q), torch.from_numpy(K)
    logits = 0.3 * (q @ k.transpose(-1, -2))
    mask = torch.ones(L, L, dtype=torch.bool).tril()
    attn = torch.softmax(logits.masked_fill(~mask, float("-inf")), dim=-1)
    np.testing.assert_allclose(F, attn.sum(dim=-2).numpy(), rtol=1e-11, atol=1e-14)


def test_zero_queries_closed_form():
    """Q = 0 makes every visible logit 0: row i is uniform over keys 0..p_i, so
    F[j] = sum over proxies with p_i >= j of 1 / (p_i + 1)."""
    L, D = 50, 4
    pos = [3, 10, 11, 30, 49]
    Q = np.zeros((1, 1, L, D))
    K = _rand((1, 1, L, D), 11)
    F, lse = proxy_scores(Q, K, pos, 1.0)
    ref = np.array([sum(1.0 / (p + 1) for p in pos if p >= j) for j in range(L)])
    np.testing.assert_allclose(F[0, 0], ref, rtol=1e-13)
    np.testing.assert_allclose(lse[0, 0], np.log(np.array(pos) + 1.0), rtol=1e-13)


def test_equal_keys_closed_form():
    """All keys equal: logits are constant per row, the same closed form holds."""
    L, D = 40, 6
    pos = [0, 9, 39]
    Q = _rand((1, 1, L, D), 12)
    K = np.broadcast_to(_rand((1, 1, 1, D), 13), (1, 1, L, D)).copy()
    F, _ = proxy_scores(Q, K, pos, 0.5)
    ref = np.array([sum(1.0 / (p + 1) for p in pos if p >= j) for j in range(L)])
    np.testing.assert_allclose(F[0, 0], ref, rtol=1e-12)


def test_key_shift_invariance():
    """Adding one vector to every key adds a per-row constant to the logits;
    row-wise softmax ignores it (fails if normalisation ran over the wrong
    axis)."""
    L, D = 80, 8
    pos = [20, 50, 79]
    Q = _rand((1, 2, L, D), 14)
    K = _rand((1, 2, L, D), 15)
    c = _rand((1, 2, 1, D), 16) * 3
    F1, _ = proxy_scores(Q, K, pos, 0.4)
    F2, _ = proxy_scores(Q, K + c, pos, 0.4)
    np.testing.assert_allclose(F1, F2, rtol=1e-10, atol=1e-14)


def test_hard_attention_limit():
    """At a huge scale each row's softmax collapses onto its largest visible
    logit, so F[j] counts the proxies whose argmax is j."""
    L, D = 30, 5
    pos = [5, 12, 20, 29]
    Q = _rand((1, 1, L, D), 17)
    K = _rand((1, 1, L, D), 18)
    F, _ = proxy_scores(Q, K, pos, 1e6)
    ref = np.zeros(L)
    for p in pos:
        ref[int(np.argmax(Q[0, 0, p] @ K[0, 0, : p + 1].T))] += 1
    np.testing.assert_allclose(F[0, 0], ref, atol=1e-9)


def test_lse_matches_library_logsumexp():
    L, D = 70, 8
    pos = [10, 33, 69]
    Q = _rand((2, 1, L, D), 19)
    K = _rand((2, 1, L, D), 20)
    _, lse = proxy_scores(Q, K, pos, 0.25)
    for b in range(2):
        for i, p in enumerate(pos):
            a = 0.25 * (Q[b, 0, p] @ K[b, 0, : p + 1].T)
            assert abs(lse[b, 0, i] - scipy.special.logsumexp(a)) < 1e-12


def test_scale_enters_logits():
    """Doubling the scale equals doubling the queries."""
    L, D = 40, 4
    pos = [17, 39]
    Q = _rand((1, 1, L, D), 21)
    K = _rand((1, 1, L, D), 22)
    F1, _ = proxy_scores(Q, K, pos, 0.6)
    F2, _ = proxy_scores(2 * Q, K, pos, 0.3)
    np.testing.assert_allclose(F1, F2, rtol=1e-12)


def test_bf16_inputs_convert_exactly():
    """bf16 values enter the float64 arithmetic unchanged."""
    L, D = 32, 8
    q = torch.randn(1, 1, L, D).to(torch.bfloat16)
    k = torch.randn(1, 1, L, D).to(torch.bfloat16)
    F1, _ = proxy_scores(q.float().numpy(), k.float().numpy(), [31], 0.5)
    F2, _ = proxy_scores(q.double().numpy(), k.double().numpy(), [31], 0.5)
    assert np.array_equal(F1, F2)
