"""GPU parity of the prefill's causal attention and its per-row log-sum-exp
(the forward pass whose log-sum-exp Appendix A.7 hands to the score), and of
the single-pass score (Algorithm 2) fed with that log-sum-exp.

Tolerances, from the arithmetic: logits are exact bf16 products summed in
fp32, and the row sums and the log-sum-exp stay in fp32, so the log-sum-exp
is held to 1e-4 absolute.  The output rounds each probability to bf16
(relative error at most 2^-9) before the value product and the finished row
to bf16 once more, so |O - O_ref| <= 2^-9 max|V| + 2^-9 |O_ref| <= 2^-8 max|V|;
the test allows 4.5e-3 max|V|."""

import sys

import numpy as np
import pytest
import torch

from oracle import causal_attention, proxy_scores_grouped
from synth import custom, make_grouped_layer, make_layer
from tests._parity import check_scores

pytestmark = pytest.mark.gpu

nacl = pytest.importorskip("paper_2408_03675_amd.nacl")

LSE_ATOL = 1e-4
O_TOL = 4.5e-3  # times max|V|


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nacl.load_library()


def _f64(t):
    return t.detach().cpu().double().numpy()


def _check(out, lse, q, k, v, s, g, label, rows=None):
    Or, lr = causal_attention(_f64(q), _f64(k), _f64(v), s, q_group=g, rows=rows)
    o = _f64(out) if rows is None else _f64(out[:, :, rows])
    l = _f64(lse) if rows is None else _f64(lse[:, :, rows])
    assert np.isfinite(o).all() and np.isfinite(l).all(), label
    vmax = float(_f64(v).__abs__().max())
    err_o = np.abs(o - Or).max()
    err_l = np.abs(l - lr).max()
    assert err_o <= O_TOL * vmax, f"{label}: output off by {err_o} (max|V| {vmax})"
    assert err_l <= LSE_ATOL, f"{label}: log-sum-exp off by {err_l}"
    return err_o / vmax, err_l


CASES = [
    # name, B, H (K/V heads), q_group, L, D, injected sinks and heavy hitters
    ("d128_ragged300", 1, 2, 1, 300, 128, False),
    ("d64_ragged257", 2, 2, 1, 257, 64, False),
    ("gqa4_d128_640", 1, 2, 4, 640, 128, False),
    ("one_row", 1, 1, 1, 1, 128, False),
    ("one_tile64", 1, 3, 1, 64, 128, False),
    ("tiles_129", 1, 1, 2, 129, 64, False),
    ("sinks_1000", 1, 2, 1, 1000, 128, True),
    ("sinks_d64_777", 2, 1, 1, 777, 64, True),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_attention_matches_oracle(case):
    name, B, H, g, L, D, inject = case
    print("attention case", name, file=sys.stderr, flush=True)
    P = max(1, L // 50)
    w = custom(name, B, H, L, D, P, dtype="bf16", inject=inject, data_seed=len(name) * 11)
    q, k, v = make_grouped_layer(w, g, device="cuda") if g > 1 else make_layer(w, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos)
    out, lse, _ = nacl.attention(prob, q, k, v)
    torch.cuda.synchronize()
    _check(out, lse, q, k, v, prob.c.sm_scale, g, name)


def test_attention_strided_layout():
    """Q, K, V as [B, L, H, D] buffers viewed as [B, H, L, D] (row stride H * D)."""
    B, H, g, L, D = 2, 2, 2, 333, 128
    gen = torch.Generator(device="cuda")
    gen.manual_seed(5)
    qb = torch.randn((B, L, H * g, D), generator=gen, device="cuda").to(torch.bfloat16)
    kb = torch.randn((B, L, H, D), generator=gen, device="cuda").to(torch.bfloat16)
    vb = torch.randn((B, L, H, D), generator=gen, device="cuda").to(torch.bfloat16)
    q, k, v = qb.transpose(1, 2), kb.transpose(1, 2), vb.transpose(1, 2)
    pos = list(range(7, L, 41))
    prob = nacl.Problem.from_tensors(q, k, v, pos)
    out, lse, _ = nacl.attention(prob, q, k, v)
    torch.cuda.synchronize()
    _check(out, lse, q, k, v, prob.c.sm_scale, g, "strided")


@pytest.mark.parametrize("g", [1, 4])
def test_single_pass_score_from_attention_lse(g):
    """Appendix A.7's pipeline: the attention's log-sum-exp at the proxy rows
    feeds the score's column reduction (Algorithm 2), which must give the
    oracle's F; the gathered rows must equal the full log-sum-exp's."""
    B, H, L, D, P = 2, 2, 2500, 128, 40
    w = custom(f"a7_{g}", B, H, L, D, P, dtype="bf16", inject=(g == 1), data_seed=77 + g)
    q, k, v = make_grouped_layer(w, g, device="cuda") if g > 1 else make_layer(w, device="cuda")
    pos_dev = torch.tensor(w.proxy_pos, dtype=torch.int32, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos, proxy_pos_dev=pos_dev)
    out, lse, lp = nacl.attention(prob, q, k, v, lse_proxy=True)
    F = nacl.score(prob, q, k, nacl.workspace(prob), lse=lp)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(lp.cpu().numpy(), lse[:, :, w.proxy_pos].cpu().numpy())
    Fr, lr = proxy_scores_grouped(_f64(q), _f64(k), w.proxy_pos, prob.c.sm_scale, g)
    assert np.abs(_f64(lp) - lr).max() <= LSE_ATOL
    check_scores(F.cpu().numpy(), Fr, f"a7_g{g}")


def test_attention_prefill_32k_sampled_rows():
    """The 32k prefill layer at full size (B = 4, H = 32, L = 32768, D = 128,
    bf16, injected sinks and heavy hitters): every row's log-sum-exp is
    finite, and sampled rows of sampled heads match the oracle."""
    B, H, L, D, P = 4, 32, 32768, 128, 128
    w = custom("prefill_32k_attention", B, H, L, D, P, dtype="bf16", inject=True, data_seed=3)
    q, k, v = make_layer(w, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos)
    out, lse, _ = nacl.attention(prob, q, k, v)
    torch.cuda.synchronize()
    assert torch.isfinite(lse).all()
    rows = np.array([0, 1, 127, 128, 4095, 16384, 32766, 32767])
    for b, h in ((0, 0), (1, 17), (3, 31)):
        sl = slice(h, h + 1)
        _check(out[b:b + 1, sl], lse[b:b + 1, sl], q[b:b + 1, sl], k[b:b + 1, sl], v[b:b + 1, sl],
               prob.c.sm_scale, 1, f"32k b{b} h{h}", rows=rows)


def test_attention_d64_grouped_4k_sampled_rows():
    """Head dim 64 with two query heads per K/V head over 4097 tokens (33
    query tiles of 128 rows per head, the last holding one row): sampled rows
    of every head, and every log-sum-exp finite."""
    B, H, g, L, D, P = 2, 4, 2, 4097, 64, 64
    w = custom("gqa_d64_4k", B, H, L, D, P, dtype="bf16", data_seed=41)
    q, k, v = make_grouped_layer(w, g, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos)
    out, lse, _ = nacl.attention(prob, q, k, v)
    torch.cuda.synchronize()
    assert torch.isfinite(lse).all()
    rows = np.array([0, 63, 64, 127, 128, 255, 256, 2048, 4095, 4096])
    _check(out, lse, q, k, v, prob.c.sm_scale, g, "gqa_d64_4k", rows=rows)


@pytest.mark.parametrize("L,g,scale", [(128, 1, 0.05), (256, 8, None), (2, 1, 2.0)])
def test_attention_tile_multiples_and_scales(L, g, scale):
    """Exact multiples of the 128-row and 64-key tiles, eight query heads per
    K/V head, two rows, and logit scales other than 1/sqrt(D)."""
    B, H, D = 1, 2, 128
    w = custom(f"edge_{L}_{g}", B, H, L, D, 1, dtype="bf16", data_seed=L + g)
    q, k, v = make_grouped_layer(w, g, device="cuda") if g > 1 else make_layer(w, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos, sm_scale=scale)
    out, lse, _ = nacl.attention(prob, q, k, v)
    torch.cuda.synchronize()
    _check(out, lse, q, k, v, prob.c.sm_scale, g, f"edge L{L} g{g}")


def test_attention_rejects_unsupported():
    q = torch.zeros((1, 1, 16, 64), dtype=torch.float32, device="cuda")
    prob = nacl.Problem.from_tensors(q, q, q, [3])
    with pytest.raises(nacl.NaclError) as e:
        nacl.attention(prob, q, q, q, out=torch.empty_like(q))
    assert e.value.status == 2
    qb = torch.zeros((1, 1, 16, 64), dtype=torch.bfloat16, device="cuda")
    prob = nacl.Problem.from_tensors(qb, qb, qb, [3])
    with pytest.raises(nacl.NaclError):
        nacl.attention(prob, qb, qb, qb, lse_proxy=True)  # no proxy_pos_dev
