"""GPU parity: the HIP library through its C ABI against the CPU oracle.

Small problems run whole through the oracle (several tiles, ragged tails,
scattered and multi-group proxies, fp32 and bf16, D = 64 and 128, strided
inputs).  Bars: scores within 1e-3 relative; isolated selection on identical
fp32 scores exactly equal; end-to-end keep sets equal up to near-ties;
compacted rows bit-exact.
"""

import sys
import zlib
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import (SAMPLE_PROPORTIONAL, SAMPLE_SOFTMAX, SAMPLE_UNIFORM, compact as o_compact,
                    proxy_scores, select_head)
from synth import WORKLOADS, custom, make_layer
from tests._parity import (check_keep_near, check_keep_valid, check_rows_for_common,
                           check_scores)

pytestmark = pytest.mark.gpu

nacl = pytest.importorskip("paper_2408_03675_amd.nacl")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nacl.load_library()


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _np(t):
    return t.detach().float().cpu().numpy() if t.dtype == torch.bfloat16 else t.detach().cpu().numpy()


def _layer(w, device="cuda"):
    q, k, v = make_layer(w, 0, device=device)
    return q, k, v


SCORE_CASES = [
    # name, B, H, L, D, dtype, positions
    ("f32_d64_suffix", 1, 4, 2048, 64, "f32", list(range(2016, 2048))),
    ("bf16_d128_ragged", 2, 3, 1000, 128, "bf16", list(range(900, 1000))),
    ("bf16_d64_scattered", 2, 2, 1037, 64, "bf16", [0, 5, 17, 300, 301, 302, 640, 1000, 1036]),
    ("f32_d128_scattered", 1, 2, 777, 128, "f32", sorted(set(range(3, 777, 21)))),
    ("bf16_all_tokens", 1, 2, 96, 64, "bf16", list(range(96))),
    ("bf16_multigroup", 1, 2, 530, 128, "bf16", list(range(330, 530))),
    ("f32_single_proxy_mid", 1, 1, 2049, 128, "f32", [1500]),
    ("bf16_len1", 1, 1, 1, 64, "bf16", [0]),
    ("bf16_len17", 2, 1, 17, 128, "bf16", [16]),
    # the proxy-split kernel (bf16, D = 128, P >= 128): scattered proxies over several
    # 2048-key items with a ragged tail, and proxies early so later items lie past them
    ("bf16_split_scattered", 1, 2, 5001, 128, "bf16", sorted(set(range(7, 5001, 31)))),
    ("bf16_split_early", 2, 1, 4100, 128, "bf16", list(range(200, 330))),
    # exactly 128 proxies (the benchmark's proxy count): a ragged tail, scattered
    # proxies, items past the last proxy, proxies at the start
    ("bf16_p128_suffix", 2, 3, 1000, 128, "bf16", list(range(872, 1000))),
    ("bf16_p128_scattered", 1, 2, 5001, 128, "bf16", [7 + 39 * i for i in range(128)]),
    ("bf16_p128_early", 2, 1, 4100, 128, "bf16", list(range(200, 328))),
    ("bf16_p128_first", 1, 3, 300, 128, "bf16", list(range(128))),
    # more than 512 proxies: the wide proxy-split kernel over two and three groups of 512
    # (column sums accumulated across groups), and the per-wave-tile kernel for fp32
    ("bf16_wide_two_groups", 1, 2, 3000, 128, "bf16", sorted(set(range(5, 3000, 5)))),
    ("bf16_wide_three_groups", 1, 1, 2300, 128, "bf16", list(range(1200, 2300))),
    ("f32_many_proxies", 1, 2, 1500, 64, "f32", list(range(800, 1500))),
    ("bf16_d64_three_groups", 1, 2, 1200, 64, "bf16", list(range(900, 1200))),
    # few proxy rows (K read once, logits kept): one row at the last token over several
    # 512-key chunks with a ragged tail, the most rows each element size takes, rows whose
    # positions leave whole chunks unseen, and a head shorter than one tile
    ("bf16_rows_last_token", 2, 3, 6617, 128, "bf16", [6616]),
    ("bf16_rows16_spread", 1, 2, 5001, 128, "bf16", [40 + 311 * i for i in range(16)]),
    ("bf16_d64_rows8", 2, 2, 1500, 64, "bf16", [3, 100, 511, 512, 513, 900, 1400, 1499]),
    ("f32_d64_rows16", 1, 2, 2049, 64, "f32", list(range(700, 716))),
    ("f32_d128_rows_early", 2, 1, 3000, 128, "f32", [10, 20, 600]),
    ("bf16_rows_short", 1, 2, 13, 128, "bf16", [2, 12]),
]


@pytest.mark.parametrize("case", SCORE_CASES, ids=[c[0] for c in SCORE_CASES])
def test_score_matches_oracle(case):
    name, B, H, L, D, dt, pos = case
    _say("score case", name)
    w = custom(name, B, H, L, D, len(pos), dtype=dt, data_seed=zlib.crc32(name.encode()) % 1000)
    q, k, v = make_layer(w, 0, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, pos)
    ws = nacl.workspace(prob)
    F = nacl.score(prob, q, k, ws)
    torch.cuda.synchronize()
    Fr, _ = proxy_scores(_np(q), _np(k), pos, prob.c.sm_scale)
    rel = check_scores(F.cpu().numpy(), Fr, name)
    np.testing.assert_allclose(F.cpu().numpy().astype(np.float64).sum(-1), len(pos), rtol=1e-5)
    _say("  max rel err", rel)


@pytest.mark.parametrize("pos", [list(range(650, 700)), [10, 350, 699]], ids=["p50", "few_rows"])
def test_score_strided_inputs(pos):
    """Q, K, V as [B, H, L, D] views of [B, L, H, D] buffers (50 proxies, and
    three: the few-row path)."""
    B, H, L, D = 2, 4, 700, 128
    g = torch.Generator(device="cuda").manual_seed(7)
    base = torch.randn((3, B, L, H, D), generator=g, device="cuda").to(torch.bfloat16)
    q, k, v = (base[i].permute(0, 2, 1, 3) for i in range(3))
    prob = nacl.Problem.from_tensors(q, k, v, pos)
    ws = nacl.workspace(prob)
    F = nacl.score(prob, q, k, ws)
    Fr, _ = proxy_scores(_np(q), _np(k), pos, prob.c.sm_scale)
    check_scores(F.cpu().numpy(), Fr, "strided")


@pytest.mark.parametrize("P", [3, 40, 160, 700])
def test_score_with_caller_lse(P):
    """With the caller's log-sum-exp (Appendix A.7, Algorithm 2) only the
    column reduction runs and gives the same scores (P = 3: a few-row problem,
    which with a caller LSE takes the per-wave-tile kernel's single pass;
    P = 160: the proxy-split kernel, a full and a partial proxy group; P = 700:
    the wide kernel, a full and a partial group of 512)."""
    w = custom("lse", 1, 3, 1500, 128, P, dtype="bf16", data_seed=3)
    q, k, v = make_layer(w, 0, device="cuda")
    pos = w.proxy_pos
    prob = nacl.Problem.from_tensors(q, k, v, pos)
    Fr, lse = proxy_scores(_np(q), _np(k), pos, prob.c.sm_scale)
    lse_t = torch.from_numpy(lse.astype(np.float32)).cuda()
    F = nacl.score(prob, q, k, nacl.workspace(prob), lse=lse_t)
    check_scores(F.cpu().numpy(), Fr, "caller lse")


@pytest.mark.parametrize("P", [100, 128, 160, 600])
def test_score_overflow_takes_exact_path(P):
    """Pass 1 sums exp2(logit - r) against the maximum r of the first tile of
    each item's key range; a later key far above r overflows fp32, and the
    kernel recomputes that range's sums against its exact maximum.  Here one
    key per head sits about 180 (natural-log units) above every other logit
    of its range, so the fast path overflows and the scores are dominated by
    that key (P = 100: the per-wave-tile kernel; P = 128 and 160: the
    proxy-split kernel; P = 600: its wide form)."""
    B, H, L, D = 1, 2, 3000, 128
    g = torch.Generator(device="cuda").manual_seed(11)
    q = torch.randn((B, H, L, D), generator=g, device="cuda")
    k = torch.randn((B, H, L, D), generator=g, device="cuda")
    pos = list(range(L - P, L))
    q[:, :, L - P:] += 2.0       # proxy rows with a positive mean
    k[:, 0, 1000] = 8.0          # head 0: a key inside a range, not in its first tile
    k[:, 1, 2500] = 8.0          # head 1: the same in another item
    q, k = q.to(torch.bfloat16), k.to(torch.bfloat16)
    prob = nacl.Problem.from_tensors(q, k, k, pos)
    F = nacl.score(prob, q, k, nacl.workspace(prob))
    torch.cuda.synchronize()
    Fr, _ = proxy_scores(_np(q), _np(k), pos, prob.c.sm_scale)
    check_scores(F.cpu().numpy(), Fr, "overflow")
    for h, j in ((0, 1000), (1, 2500)):  # nearly all the mass of every proxy that sees key j
        assert float(F[0, h, j]) > 0.99 * sum(p >= j for p in pos)


def test_score_config_small_and_longbench():
    for key in ("small_f32", "longbench_4k"):
        w = WORKLOADS[key]
        _say("score workload", key)
        q, k, v = _layer(w)
        prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos, sm_scale=w.scale)
        F = nacl.score(prob, q, k, nacl.workspace(prob))
        Fr, _ = proxy_scores(_np(q), _np(k), w.proxy_pos, w.scale)
        check_scores(F.cpu().numpy(), Fr, key)


SELECT_CASES = [
    # name, L, P, n_protect, C, Cr, mode, ties
    ("softmax_basic", 2048, 32, 32, 409, 245, SAMPLE_SOFTMAX, False),
    ("proportional", 3001, 50, 50, 600, 200, SAMPLE_PROPORTIONAL, False),
    ("uniform", 1000, 10, 10, 300, 150, SAMPLE_UNIFORM, False),
    ("no_random", 4096, 64, 64, 819, 0, SAMPLE_SOFTMAX, False),
    ("all_random", 4096, 64, 64, 819, 755, SAMPLE_SOFTMAX, False),
    ("no_protect", 1500, 20, 0, 300, 100, SAMPLE_SOFTMAX, False),
    ("keep_all", 777, 7, 7, 777, 300, SAMPLE_SOFTMAX, False),
    ("keep_protected_only", 512, 16, 16, 16, 0, SAMPLE_SOFTMAX, False),
    ("ties_heavy", 5000, 8, 8, 1000, 300, SAMPLE_SOFTMAX, True),
    ("ties_uniform", 2500, 8, 4, 700, 100, SAMPLE_UNIFORM, True),
    ("tiny", 5, 1, 1, 3, 1, SAMPLE_SOFTMAX, False),
    ("empty_budget", 100, 4, 0, 0, 0, SAMPLE_SOFTMAX, False),
    # long heads (keys held in registers up to 32k tokens), ties, extreme budgets
    ("long_softmax", 20000, 128, 128, 4000, 2000, SAMPLE_SOFTMAX, False),
    ("long_proportional", 9001, 40, 20, 1800, 600, SAMPLE_PROPORTIONAL, False),
    ("long_uniform", 12288, 64, 64, 2457, 1228, SAMPLE_UNIFORM, False),
    ("long_ties", 16384, 16, 16, 3000, 1000, SAMPLE_SOFTMAX, True),
    ("long_small_budget", 32768, 128, 128, 400, 100, SAMPLE_SOFTMAX, False),
    ("long_large_budget", 32768, 128, 128, 30000, 20000, SAMPLE_SOFTMAX, False),
]


@pytest.mark.parametrize("case", SELECT_CASES, ids=[c[0] for c in SELECT_CASES])
def test_select_exact_on_identical_scores(case):
    name, L, P, n_protect, C, Cr, mode, ties = case
    _say("select case", name)
    B, H = 2, 3
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    F = rng.gamma(0.3, 1.0 / L, size=(B, H, L))
    if ties:
        F = np.round(F * L * 4) / (L * 4)
    F32 = F.astype(np.float32)
    pos = list(range(L - P, L))
    prob = nacl.Problem(B, H, L, 128, "bf16", pos, n_protect=n_protect)
    ws = nacl.workspace(prob)
    keep = nacl.select(prob, torch.from_numpy(F32).cuda(), C, Cr, mode, seed=1234, layer=5, ws=ws)
    keep = keep.cpu().numpy()
    for b in range(B):
        for h in range(H):
            ref = select_head(F32[b, h], pos, n_protect, C, Cr, mode, 1234, 5, b, h)
            assert np.array_equal(keep[b, h], ref["keep"]), (name, b, h)


LONG_SELECT_CASES = [
    # heads longer than 32768 tokens (one work-group per 16384-token slice):
    # ties, odd lengths, tiny and near-total budgets, no or only random tokens
    # name, L, P, n_protect, C, Cr, mode, ties
    ("long_ties_65k", 65536, 64, 64, 13107, 6553, SAMPLE_SOFTMAX, True),
    ("odd_40001", 40001, 17, 17, 8000, 3000, SAMPLE_PROPORTIONAL, False),
    ("small_k_100k", 100000, 128, 128, 300, 100, SAMPLE_SOFTMAX, False),
    ("large_budget_70k", 70000, 32, 32, 69000, 30000, SAMPLE_SOFTMAX, False),
    ("uniform_ties_50k", 50000, 64, 32, 10000, 5000, SAMPLE_UNIFORM, True),
    ("no_random_33k", 32769, 16, 16, 6000, 0, SAMPLE_SOFTMAX, False),
    ("all_random_45k", 45000, 16, 16, 9000, 8984, SAMPLE_SOFTMAX, False),
    ("keep_all_36k", 36000, 8, 8, 36000, 10000, SAMPLE_SOFTMAX, False),
    ("heavy_ties_128k", 131072, 512, 512, 26214, 15728, SAMPLE_SOFTMAX, True),
]


@pytest.mark.parametrize("case", LONG_SELECT_CASES, ids=[c[0] for c in LONG_SELECT_CASES])
def test_select_exact_long_heads(case):
    name, L, P, n_protect, C, Cr, mode, ties = case
    _say("long select case", name)
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    F = rng.gamma(0.3, 1.0 / L, size=(1, 2, L))
    if ties:
        F = np.round(F * L * 4) / (L * 4)
    F32 = F.astype(np.float32)
    pos = list(range(L - P, L))
    prob = nacl.Problem(1, 2, L, 128, "bf16", pos, n_protect=n_protect)
    ws = nacl.workspace(prob)
    keep = nacl.select(prob, torch.from_numpy(F32).cuda(), C, Cr, mode, seed=1234, layer=5, ws=ws)
    keep = keep.cpu().numpy()
    assert nacl.health(ws) == (0, 0)
    for h in range(2):
        ref = select_head(F32[0, h], pos, n_protect, C, Cr, mode, 1234, 5, 0, h)
        assert np.array_equal(keep[0, h], ref["keep"]), (name, h)


def test_select_full_length_limit_head():
    """A long head (131072 tokens, the 128k workload's length)."""
    L, P, C, Cr = 131072, 512, 26214, 15728
    rng = np.random.default_rng(9)
    F32 = rng.gamma(0.5, 512.0 / L / 0.5, size=(1, 2, L)).astype(np.float32)
    pos = list(range(L - P, L))
    prob = nacl.Problem(1, 2, L, 128, "bf16", pos)
    keep = nacl.select(prob, torch.from_numpy(F32).cuda(), C, Cr, SAMPLE_SOFTMAX, 0, 0,
                       ws=nacl.workspace(prob)).cpu().numpy()
    for h in range(2):
        ref = select_head(F32[0, h], pos, P, C, Cr, SAMPLE_SOFTMAX, 0, 0, 0, h)
        assert np.array_equal(keep[0, h], ref["keep"])


@pytest.mark.parametrize("dt,D", [("bf16", 128), ("bf16", 64), ("f32", 64), ("f32", 128)])
def test_compact_bit_exact(dt, D):
    B, H, L, C = 2, 3, 1000, 211
    w = custom("cmp", B, H, L, D, 4, dtype=dt, data_seed=D)
    q, k, v = make_layer(w, 0, device="cuda")
    rng = np.random.default_rng(D)
    idx = np.sort(np.stack([[rng.choice(L, C, replace=False) for _ in range(H)] for _ in range(B)]), -1)
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos)
    ko, vo = nacl.compact(prob, k, v, torch.from_numpy(idx.astype(np.int32)).cuda())
    kr, vr = o_compact(k.cpu().view(torch.int16 if dt == "bf16" else torch.int32).numpy(),
                       v.cpu().view(torch.int16 if dt == "bf16" else torch.int32).numpy(), idx)
    view = torch.int16 if dt == "bf16" else torch.int32
    assert np.array_equal(ko.cpu().view(view).numpy(), kr)
    assert np.array_equal(vo.cpu().view(view).numpy(), vr)


def _evict_and_compare(w, layer=0, heads=None, keep_frac=None, random_share=None, label=""):
    q, k, v = make_layer(w, layer, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos, sm_scale=w.scale)
    ws = nacl.workspace(prob)
    F, keep, ko, vo = nacl.evict(prob, q, k, v, w.C, w.Cr, SAMPLE_SOFTMAX, w.rng_seed, layer, ws=ws)
    torch.cuda.synchronize()
    F = F.cpu().numpy()
    keep = keep.cpu().numpy()
    check_keep_valid(keep, w.L, w.C, w.proxy_pos[w.P - w.n_protect:])
    np.testing.assert_allclose(F.astype(np.float64).sum(-1), w.P, rtol=1e-5)
    if heads is None:
        heads = [(b, h) for b in range(w.B) for h in range(w.H)]
    view = torch.int16 if w.dtype == "bf16" else torch.int32
    n_diff = 0
    for (b, h) in heads:
        qh = _np(q[b:b + 1, h:h + 1])
        kh = _np(k[b:b + 1, h:h + 1])
        Fr, _ = proxy_scores(qh, kh, w.proxy_pos, w.scale)
        check_scores(F[b, h], Fr[0, 0], f"{label} F b={b} h={h}")
        Fr32 = Fr[0, 0].astype(np.float32)
        ref = select_head(Fr32, w.proxy_pos, w.n_protect, w.C, w.Cr, SAMPLE_SOFTMAX, w.rng_seed,
                          layer, b, h)
        n_diff += check_keep_near(keep[b, h], ref, Fr32, w.Cr, f"{label} keep b={b} h={h}")
        kbits = k[b, h].cpu().view(view).numpy()
        vbits = v[b, h].cpu().view(view).numpy()
        check_rows_for_common(keep[b, h], ko[b, h].cpu().view(view).numpy(), ref["keep"],
                              kbits[ref["keep"]], f"{label} K' b={b} h={h}")
        check_rows_for_common(keep[b, h], vo[b, h].cpu().view(view).numpy(), ref["keep"],
                              vbits[ref["keep"]], f"{label} V' b={b} h={h}")
    _say(f"  {label}: {len(heads)} heads compared, {n_diff} near-tie differences")


def test_evict_small_f32_all_heads():
    _evict_and_compare(WORKLOADS["small_f32"], label="small_f32")


def test_evict_longbench_all_heads():
    _evict_and_compare(WORKLOADS["longbench_4k"], label="longbench_4k")


def test_evict_empty_budget():
    """C = 0 (nothing kept, no proxy protected): the scores are still computed, the keep
    set and the compacted cache are empty."""
    w = custom("empty", 1, 2, 600, 128, 8, dtype="bf16", data_seed=4)
    q, k, v = make_layer(w, 0, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos, n_protect=0)
    F, keep, ko, vo = nacl.evict(prob, q, k, v, 0, 0, SAMPLE_SOFTMAX, 0, 0, ws=nacl.workspace(prob))
    torch.cuda.synchronize()
    assert tuple(keep.shape) == (1, 2, 0) and tuple(ko.shape) == (1, 2, 0, 128) and ko.numel() == 0
    Fr, _ = proxy_scores(_np(q), _np(k), w.proxy_pos, prob.c.sm_scale)
    check_scores(F.cpu().numpy(), Fr, "empty budget")


def test_evict_many_protected_proxies():
    """599 proxies, all protected (the wide score kernel over two groups of 512; the
    selection excludes 599 tokens from both draws): scores, keep sets and compacted rows
    against the oracle on every head."""
    w = custom("evict_many_proxies", 1, 2, 3000, 128, 599, keep_frac=Fraction(1, 2),
               random_share=Fraction(1, 5), inject=True, data_seed=17)
    _evict_and_compare(w, label="many proxies")


def test_evict_is_deterministic():
    w = WORKLOADS["longbench_4k"]
    q, k, v = make_layer(w, 0, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos)
    ws = nacl.workspace(prob)
    a = [t.clone() for t in nacl.evict(prob, q, k, v, w.C, w.Cr, 0, 7, 3, ws=ws)]
    b = nacl.evict(prob, q, k, v, w.C, w.Cr, 0, 7, 3, ws=ws)
    for x, y in zip(a, b):
        assert torch.equal(x, y)
    c = nacl.evict(prob, q, k, v, w.C, w.Cr, 0, 7, 4, ws=ws)
    assert not torch.equal(a[1], c[1])


@pytest.mark.parametrize("mode", [SAMPLE_SOFTMAX, SAMPLE_PROPORTIONAL, SAMPLE_UNIFORM])
@pytest.mark.parametrize("where", ["end", "early"])
@pytest.mark.parametrize("P", [1, 6, 40, 128, 160])
def test_evict_draws_the_same_keys_as_select(mode, where, P):
    """nacl_evict draws the Gumbel keys inside the column reduction (skipping
    the selection's key kernel); its keep set must equal that of nacl_select
    run on the same scores, which draws every key in its own kernel.  Proxies
    at the end, or early so that whole chunks lie past the last proxy (scores
    0, keys drawn on the zero path); L not a multiple of 4; every non-protected
    slot random, so every key's value matters.  P = 160 runs the proxy-split
    score kernel on one proxy group (P = 128) and on a full and a partial group
    (P = 160), P = 40 the per-wave-tile one, P = 1 and 6 the few-row path
    (keys drawn by its column kernel)."""
    B, H, L, D = 2, 3, 9001, 128
    pos = list(range(L - P, L)) if where == "end" else list(range(300, 300 + P))
    _say("evict keys", mode, where, P)
    w = custom("keys", B, H, L, D, len(pos), dtype="bf16", data_seed=61)
    q, k, v = make_layer(w, 0, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, pos)
    C = 1800
    for Cr in (C - len(pos), 700):
        F, keep, _, _ = nacl.evict(prob, q, k, v, C, Cr, mode, 11, 2, ws=nacl.workspace(prob))
        keep2 = nacl.select(prob, F, C, Cr, mode, 11, 2, ws=nacl.workspace(prob))
        torch.cuda.synchronize()
        assert torch.equal(keep, keep2), (mode, where, Cr)


def test_binding_refuses_mismatched_tensors():
    """Wrong output shapes, dtypes or input strides raise before any launch."""
    w = custom("binding", 1, 2, 300, 128, 8, dtype="bf16", data_seed=6)
    q, k, v = make_layer(w, 0, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos)
    ws = nacl.workspace(prob)
    with pytest.raises(ValueError, match="shape"):
        nacl.score(prob, q, k, ws, out=torch.empty((1, 2, 299), device="cuda"))
    with pytest.raises(ValueError, match="dtype"):
        nacl.select(prob, torch.zeros((1, 2, 300), device="cuda", dtype=torch.float64), 60, 10, ws=ws)
    with pytest.raises(ValueError, match="strides"):
        nacl.score(prob, q, k.transpose(1, 2).contiguous().transpose(1, 2), ws)
    with pytest.raises(ValueError, match="shape"):
        nacl.evict(prob, q, k, v, 60, 10, ws=ws, k_out=torch.empty((1, 2, 59, 128), device="cuda",
                                                                  dtype=torch.bfloat16))
    F = nacl.score(prob, q, k, ws)  # the same call with matching tensors runs
    torch.cuda.synchronize()
    assert torch.isfinite(F).all()
