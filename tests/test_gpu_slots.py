"""GPU parity of the slot form of the generation-phase cache update
(Section 3, "Generation Phase Eviction"): kept rows below C stay in their
slots and the kept rows at or past C fill the other slots below C, both in
ascending order (the oracle's slot_layout).  The slot layout is integer work
and is compared exactly; rows are compared bit for bit; rows at or past C and
the keep list itself are left untouched.
"""

import sys

import numpy as np
import pytest
import torch

from oracle import SAMPLE_SOFTMAX, proxy_scores, select_head, slot_layout
from synth import custom, make_layer
from tests._parity import check_keep_near, check_keep_valid, check_scores

pytestmark = pytest.mark.gpu

nacl = pytest.importorskip("paper_2408_03675_amd.nacl")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nacl.load_library()


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _bits(t):
    return t.detach().cpu().view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).numpy()


def _check_layout(kb, vb, ka, va, keep, slots, C, label):
    """kb, vb: cache bits before; ka, va: after; keep: ascending keep sets;
    slots: the GPU's slot layout."""
    B, H = keep.shape[:2]
    for b in range(B):
        for h in range(H):
            want = slot_layout(keep[b, h], C)
            assert np.array_equal(slots[b, h], want), f"{label} slot layout b={b} h={h}"
            assert np.array_equal(ka[b, h, :C], kb[b, h][want]), f"{label} K rows b={b} h={h}"
            assert np.array_equal(va[b, h, :C], vb[b, h][want]), f"{label} V rows b={b} h={h}"
            assert np.array_equal(ka[b, h, C:], kb[b, h, C:]), f"{label} K rows past C b={b} h={h}"
            assert np.array_equal(va[b, h, C:], vb[b, h, C:]), f"{label} V rows past C b={b} h={h}"


CASES = [
    # name, B, H, C, m, D, dtype, strided, which keep sets
    ("bf16_decode", 2, 3, 409, 64, 128, "bf16", False, "random"),
    ("f32_d64_strided", 1, 4, 300, 37, 64, "f32", True, "random"),
    ("bf16_none_past_C", 1, 2, 500, 20, 128, "bf16", False, "first"),
    ("bf16_all_past_C", 1, 2, 64, 100, 64, "bf16", False, "last"),
    ("bf16_many_movers", 2, 2, 1000, 3000, 128, "bf16", False, "random"),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_compact_slots_matches_oracle(case):
    name, B, H, C, m, D, dt, strided, which = case
    _say("slot form case", name)
    L = C + m
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    g = torch.Generator(device="cuda").manual_seed(len(name))
    if strided:  # [B, H, L, D] views of [B, L, H, D] buffers
        k = torch.randn((B, L, H, D), generator=g, device="cuda").to(tdt).permute(0, 2, 1, 3)
        v = torch.randn((B, L, H, D), generator=g, device="cuda").to(tdt).permute(0, 2, 1, 3)
    else:
        k = torch.randn((B, H, L, D), generator=g, device="cuda").to(tdt)
        v = torch.randn((B, H, L, D), generator=g, device="cuda").to(tdt)
    rng = np.random.default_rng(len(name))
    keep = np.empty((B, H, C), dtype=np.int32)
    for b in range(B):
        for h in range(H):
            if which == "first":
                keep[b, h] = np.arange(C)
            elif which == "last":
                keep[b, h] = np.arange(L - C, L)
            else:
                keep[b, h] = np.sort(rng.choice(L, size=C, replace=False))
    keep_d = torch.from_numpy(keep).cuda()
    prob = nacl.Problem.from_tensors(k, k, v, [L - 1], n_protect=1)
    kb, vb = _bits(k), _bits(v)
    slots = nacl.compact_slots(prob, k, v, keep_d)
    torch.cuda.synchronize()
    assert np.array_equal(keep_d.cpu().numpy(), keep)          # read only
    _check_layout(kb, vb, _bits(k), _bits(v), keep, slots.cpu().numpy(), C, name)


def test_generation_rounds_slot_form():
    """An encoding-phase eviction of a 2048-token prompt to C = 409, then three
    rounds of m = 64 decoding steps with the slot form: nacl_append writes the
    new rows after the C slots, nacl_evict_slots scores the cache with the
    current token as the only (protected) proxy, selects, and moves only the
    kept rows among the m new ones into the freed slots.  Each round's scores
    and keep set are compared with the oracle on the cache it started from,
    the slot layout exactly."""
    B, H, L0, D, P0 = 1, 4, 2048, 128, 32
    C, m = 409, 64
    Cr = int(0.6 * C)
    L = C + m
    w = custom("gen_slots", B, H, L0, D, P0, dtype="bf16", data_seed=23)
    q, k, v = make_layer(w, 0, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos)
    kc = torch.zeros((B, H, L, D), dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros_like(kc)
    _, _, ko, vo = nacl.evict(prob, q, k, v, C, Cr, SAMPLE_SOFTMAX, 5, 0, ws=nacl.workspace(prob))
    kc[:, :, :C] = ko
    vc[:, :, :C] = vo
    g = torch.Generator(device="cuda").manual_seed(77)
    for rnd in range(3):
        new_k = torch.randn((B, H, m, D), generator=g, device="cuda").to(torch.bfloat16)
        new_v = torch.randn((B, H, m, D), generator=g, device="cuda").to(torch.bfloat16)
        probc = nacl.Problem.from_tensors(kc, kc, vc, [L - 1], n_protect=1)
        nacl.append(probc, kc, vc, C, new_k, new_v)
        q_cur = torch.randn((B, H, 1, D), generator=g, device="cuda").to(torch.bfloat16)
        q_view = q_cur.expand(B, H, L, D)
        probt = nacl.Problem.from_tensors(q_view, kc, vc, [L - 1], n_protect=1)
        torch.cuda.synchronize()
        kb, vb = _bits(kc), _bits(vc)
        k_before = kc.clone()
        seed = 2000 + rnd
        F, keep, slots = nacl.evict_slots(probt, q_view, kc, vc, C, Cr, SAMPLE_SOFTMAX, seed, 0,
                                          ws=nacl.workspace(probt))
        torch.cuda.synchronize()
        Fr, _ = proxy_scores(q_view.double().cpu().numpy(), k_before.double().cpu().numpy(), [L - 1],
                             probt.c.sm_scale)
        check_scores(F.cpu().numpy(), Fr, f"round {rnd} F")
        kg = keep.cpu().numpy()
        check_keep_valid(kg, L, C, [L - 1])
        n = 0
        for b in range(B):
            for h in range(H):
                Fr32 = Fr[b, h].astype(np.float32)
                ref = select_head(Fr32, [L - 1], 1, C, Cr, SAMPLE_SOFTMAX, seed, 0, b, h)
                n += check_keep_near(kg[b, h], ref, Fr32, Cr, f"round {rnd} keep b={b} h={h}",
                                     mode=SAMPLE_SOFTMAX)
        _check_layout(kb, vb, _bits(kc), _bits(vc), kg, slots.cpu().numpy(), C, f"round {rnd}")
        assert (slots.cpu().numpy() == L - 1).sum(-1).tolist() == [[1] * H] * B  # the current token stays
        _say(f"  slot-form round {rnd}: {n} near-tie differences")
