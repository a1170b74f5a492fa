"""GPU parity of the paper's variants and special cases, all through the same
C ABI the encoding-phase eviction uses.

- Generation-phase eviction (Section 3, "Generation Phase Eviction"; the
  Generation function of Algorithm 1): every m decoding steps the cache, now
  C + m entries long, is evicted back to C with the attention row of the
  current token, i.e. one proxy at the last cache position, kept by default.
  The current token's query is passed as a [B, H, 1, D] tensor viewed with a
  zero l-stride, so no [B, H, L, D] query buffer is needed.
- MSRNN special case (Section 5.1: the proxy set is the current token only).
- H2O special case (Section 5.1: the proxy set is every token).
- Proxies at the beginning and the end of the prompt (Appendix A.3).

Bars as elsewhere: scores within 1e-3 relative of the float64 oracle, keep
sets equal up to near-ties, compacted rows bit-exact.
"""

import sys

import numpy as np
import pytest
import torch

from oracle import SAMPLE_SOFTMAX, SAMPLE_UNIFORM, proxy_scores, select_head
from synth import custom, make_layer
from tests._parity import check_keep_near, check_keep_valid, check_rows_for_common, check_scores

pytestmark = pytest.mark.gpu

nacl = pytest.importorskip("paper_2408_03675_amd.nacl")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nacl.load_library()


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _f64(t):
    return t.detach().cpu().double().numpy()


def _compare_eviction(q_full, k, v, pos, n_protect, C, Cr, mode, seed, layer, scale, F, keep, ko, vo, label):
    """Element-wise comparison of one eviction call with the oracle."""
    B, H = k.shape[:2]
    Fr, _ = proxy_scores(_f64(q_full), _f64(k), pos, scale)
    check_scores(F.cpu().numpy(), Fr, f"{label} F")
    kg = keep.cpu().numpy()
    check_keep_valid(kg, k.shape[2], C, pos[len(pos) - n_protect:])
    view = torch.int16 if k.dtype == torch.bfloat16 else torch.int32
    n_diff = 0
    for b in range(B):
        for h in range(H):
            Fr32 = Fr[b, h].astype(np.float32)
            ref = select_head(Fr32, pos, n_protect, C, Cr, mode, seed, layer, b, h)
            n_diff += check_keep_near(kg[b, h], ref, Fr32, Cr, f"{label} keep b={b} h={h}", mode=mode)
            kbits = k[b, h].cpu().view(view).numpy()
            vbits = v[b, h].cpu().view(view).numpy()
            check_rows_for_common(kg[b, h], ko[b, h].cpu().view(view).numpy(), ref["keep"],
                                  kbits[ref["keep"]], f"{label} K' b={b} h={h}")
            check_rows_for_common(kg[b, h], vo[b, h].cpu().view(view).numpy(), ref["keep"],
                                  vbits[ref["keep"]], f"{label} V' b={b} h={h}")
    return n_diff


def test_generation_phase_eviction_rounds():
    """Encoding-phase eviction of a 2048-token prompt down to C = 409 into a
    decode cache of C + m rows per head, then three rounds of m = 64 decoding
    steps: nacl_append writes the 64 new K/V rows after the kept ones, and an
    in-place eviction (k_out = k, v_out = v) brings the cache back to C with
    the current token as the only proxy (kept), 60 % of the budget sampled and
    a fresh seed per round.  Each round is compared with the oracle on the
    cache contents it started from; rows C..C+m-1 are left as they were."""
    B, H, L0, D, P0 = 1, 4, 2048, 128, 32
    C, m = 409, 64
    Cr = int(0.6 * C)
    L = C + m
    w = custom("gen", B, H, L0, D, P0, dtype="bf16", data_seed=21)
    q, k, v = make_layer(w, 0, device="cuda")
    pos0 = w.proxy_pos
    prob = nacl.Problem.from_tensors(q, k, v, pos0)
    kc = torch.zeros((B, H, L, D), dtype=torch.bfloat16, device="cuda")   # the decode cache
    vc = torch.zeros_like(kc)
    ko = torch.empty((B, H, C, D), dtype=torch.bfloat16, device="cuda")
    vo = torch.empty_like(ko)
    F, keep, ko, vo = nacl.evict(prob, q, k, v, C, Cr, SAMPLE_SOFTMAX, 5, 0, ws=nacl.workspace(prob),
                                 k_out=ko, v_out=vo)
    torch.cuda.synchronize()
    _compare_eviction(q, k, v, pos0, P0, C, Cr, SAMPLE_SOFTMAX, 5, 0, prob.c.sm_scale, F, keep, ko, vo,
                      "encoding")
    kc[:, :, :C] = ko
    vc[:, :, :C] = vo
    probc = nacl.Problem.from_tensors(kc, kc, vc, [L - 1], n_protect=1)
    g = torch.Generator(device="cuda").manual_seed(99)
    view = torch.int16
    for rnd in range(3):
        new_k = torch.randn((B, H, m, D), generator=g, device="cuda").to(torch.bfloat16)
        new_v = torch.randn((B, H, m, D), generator=g, device="cuda").to(torch.bfloat16)
        nacl.append(probc, kc, vc, C, new_k, new_v)             # the m decoding steps' rows
        torch.cuda.synchronize()
        assert torch.equal(kc[:, :, C:].view(view), new_k.view(view))
        assert torch.equal(vc[:, :, C:].view(view), new_v.view(view))
        k_before, v_before = kc.clone(), vc.clone()
        q_cur = torch.randn((B, H, 1, D), generator=g, device="cuda").to(torch.bfloat16)
        q_view = q_cur.expand(B, H, L, D)                   # l-stride 0: every row is the current query
        pos = [L - 1]
        probt = nacl.Problem.from_tensors(q_view, kc, vc, pos, n_protect=1)
        assert probt.c.q_stride[2] == 0
        seed = 1000 + rnd
        F, keep, k_out, v_out = nacl.evict(probt, q_view, kc, vc, C, Cr, SAMPLE_SOFTMAX, seed, 0,
                                           ws=nacl.workspace(probt), in_place=True)
        torch.cuda.synchronize()
        assert k_out.data_ptr() == kc.data_ptr() and v_out.data_ptr() == vc.data_ptr()
        n = _compare_eviction(q_view, k_before, v_before, pos, 1, C, Cr, SAMPLE_SOFTMAX, seed, 0,
                              probt.c.sm_scale, F, keep, kc[:, :, :C], vc[:, :, :C], f"round {rnd}")
        kg = keep.cpu().numpy()
        assert (kg[..., -1] == L - 1).all()  # the current token stays
        kb = k_before.cpu().view(view).numpy()
        vb = v_before.cpu().view(view).numpy()
        for b in range(B):
            for h in range(H):   # the in-place rows are exactly the kept rows of the old cache
                assert np.array_equal(kc[b, h, :C].cpu().view(view).numpy(), kb[b, h][kg[b, h]])
                assert np.array_equal(vc[b, h, :C].cpu().view(view).numpy(), vb[b, h][kg[b, h]])
        assert torch.equal(kc[:, :, C:].view(view), k_before[:, :, C:].view(view))
        _say(f"  generation round {rnd}: cache {L} -> {C} in place, {n} near-tie differences")


def test_compact_in_place_and_out_of_range_rows():
    """nacl_compact in place on random ascending keep sets (dense moves, no
    move at all, one long shift; bf16 and fp32, D = 64 and 128) equals the
    oracle's gather of the cache it started from; an index outside [0, L)
    out of place gives a zero row."""
    from oracle import compact as o_compact
    rng = np.random.default_rng(12)
    for dt, D in (("bf16", 128), ("bf16", 64), ("f32", 128), ("f32", 64)):
        tdt = torch.bfloat16 if dt == "bf16" else torch.float32
        view = torch.int16 if dt == "bf16" else torch.int32
        B, H, L, C = 2, 3, 1500, 700
        k = torch.randn((B, H, L, D), device="cuda").to(tdt)
        v = torch.randn((B, H, L, D), device="cuda").to(tdt)
        idx = np.stack([np.stack([np.sort(rng.choice(L, C, replace=False)) for _ in range(H)]) for _ in range(B)])
        idx[0, 0] = np.arange(C)                 # nothing moves
        idx[1, 2] = np.arange(L - C, L)          # every row moves by L - C
        prob = nacl.Problem.from_tensors(k, k, v, [L - 1])
        kb, vb = k.cpu().view(view).numpy(), v.cpu().view(view).numpy()
        keep = torch.from_numpy(idx.astype(np.int32)).cuda()
        nacl.compact(prob, k, v, keep, in_place=True)
        torch.cuda.synchronize()
        kr, vr = o_compact(kb, vb, idx)
        assert np.array_equal(k[:, :, :C].cpu().view(view).numpy(), kr), (dt, D)
        assert np.array_equal(v[:, :, :C].cpu().view(view).numpy(), vr), (dt, D)
        assert np.array_equal(k[:, :, C:].cpu().view(view).numpy(), kb[:, :, C:])
    k = torch.randn((1, 1, 100, 128), device="cuda").to(torch.bfloat16)
    prob = nacl.Problem.from_tensors(k, k, k, [99])
    keep = torch.tensor([[[3, 150, 7]]], dtype=torch.int32, device="cuda")   # 150 is outside [0, 100)
    ko, vo = nacl.compact(prob, k, k.clone(), keep)
    torch.cuda.synchronize()
    assert torch.equal(ko[0, 0, 0], k[0, 0, 3]) and torch.equal(ko[0, 0, 2], k[0, 0, 7])
    assert not ko[0, 0, 1].float().abs().sum().item()


def test_msrnn_special_case_is_last_row_softmax():
    """Proxy set = the current (last) token only: F is that row's softmax
    over every key (Section 5.1, the MSRNN case), checked against
    torch.softmax in float64 on the same bf16 inputs."""
    w = custom("msrnn", 2, 3, 3001, 128, 1, dtype="bf16", data_seed=31)
    q, k, v = make_layer(w, 0, device="cuda")
    pos = [w.L - 1]
    prob = nacl.Problem.from_tensors(q, k, v, pos)
    F = nacl.score(prob, q, k, nacl.workspace(prob))
    qd, kd = q.double().cpu(), k.double().cpu()
    logits = torch.einsum("bhd,bhld->bhl", qd[:, :, -1], kd) * prob.c.sm_scale
    ref = torch.softmax(logits, dim=-1).numpy()
    check_scores(F.cpu().numpy(), ref, "msrnn")


def test_h2o_special_case_every_token_a_proxy():
    """Proxy set = every token (Section 5.1, the H2O case): F is the column sum
    of the full causal softmax; 1024 proxies run as eight groups of 128."""
    B, H, L, D = 1, 2, 1024, 128
    w = custom("h2o", B, H, L, D, L, dtype="bf16", data_seed=41)
    q, k, v = make_layer(w, 0, device="cuda")
    pos = list(range(L))
    prob = nacl.Problem.from_tensors(q, k, v, pos)
    F = nacl.score(prob, q, k, nacl.workspace(prob))
    Fr, _ = proxy_scores(_f64(q), _f64(k), pos, prob.c.sm_scale)
    check_scores(F.cpu().numpy(), Fr, "h2o")
    np.testing.assert_allclose(F.cpu().double().numpy().sum(-1), L, rtol=1e-5)


@pytest.mark.parametrize("mode", [SAMPLE_SOFTMAX, SAMPLE_UNIFORM])
def test_begin_and_end_proxies(mode):
    """Proxies protecting both the beginning and the end of the prompt
    (Appendix A.3, for when the question's position is unknown): 16 + 48
    proxies, all kept, the rest of the budget scored and sampled."""
    B, H, L, D = 2, 3, 4096, 128
    pos = list(range(16)) + list(range(L - 48, L))
    w = custom("begend", B, H, L, D, len(pos), dtype="bf16", data_seed=51)
    q, k, v = make_layer(w, 0, device="cuda")
    C = 819
    Cr = 491
    prob = nacl.Problem.from_tensors(q, k, v, pos)
    F, keep, ko, vo = nacl.evict(prob, q, k, v, C, Cr, mode, 3, 2, ws=nacl.workspace(prob))
    torch.cuda.synchronize()
    n = _compare_eviction(q, k, v, pos, len(pos), C, Cr, mode, 3, 2, prob.c.sm_scale, F, keep, ko, vo,
                          f"begin+end mode {mode}")
    kept = keep.cpu().numpy()
    for p in pos:
        assert (kept == p).any(-1).all()
    _say(f"  begin+end mode {mode}: {n} near-tie differences")
