"""GPU parity of grouped-query scoring (several query heads per K/V head; the
reading pinned in tests/test_oracle_grouped.py): each K/V head is scored by
the proxy rows of its group's query heads, then selected and compacted like
any head.  Every score kernel is covered (per-wave-tile below 128 proxy rows,
the proxy-split kernel, its wide form from 512 rows), as are a caller-given
log-sum-exp per query head and a whole eviction."""

import sys

import numpy as np
import pytest
import torch

from oracle import SAMPLE_SOFTMAX, proxy_scores_grouped, select_head
from synth import custom, make_grouped_layer
from tests._parity import check_keep_near, check_keep_valid, check_rows_for_common, check_scores

pytestmark = pytest.mark.gpu

nacl = pytest.importorskip("paper_2408_03675_amd.nacl")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nacl.load_library()


def _f64(t):
    return t.detach().cpu().double().numpy()


CASES = [
    # name, B, H (K/V heads), q_group, L, D, dtype, P
    ("split_rows192", 2, 4, 4, 3000, 128, "bf16", 48),
    ("tile_rows40_f32", 1, 2, 2, 2100, 64, "f32", 20),
    ("wide_rows640", 1, 2, 8, 2500, 128, "bf16", 80),
    ("kv8_q32_4k", 1, 8, 4, 4096, 128, "bf16", 64),
    ("tile_d64_bf16", 2, 3, 3, 1037, 64, "bf16", 30),
    # few rows (K read once, logits kept): the decode case (one proxy, the group's
    # query heads as rows), sixteen rows, fp32 with nine rows
    ("rows_decode_g4", 2, 4, 4, 3001, 128, "bf16", 1),
    ("rows16_g8", 1, 2, 8, 2000, 128, "bf16", 2),
    ("rows9_f32_d64_g3", 1, 3, 3, 1500, 64, "f32", 3),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_grouped_score_matches_oracle(case):
    name, B, H, g, L, D, dt, P = case
    print("grouped case", name, file=sys.stderr, flush=True)
    w = custom(name, B, H, L, D, P, dtype=dt, data_seed=len(name) * 7)
    q, k, v = make_grouped_layer(w, g, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos)
    assert prob.q_group == g
    F = nacl.score(prob, q, k, nacl.workspace(prob))
    torch.cuda.synchronize()
    Fr, _ = proxy_scores_grouped(_f64(q), _f64(k), w.proxy_pos, prob.c.sm_scale, g)
    check_scores(F.cpu().numpy(), Fr, name)
    np.testing.assert_allclose(F.double().sum(-1).cpu().numpy(), P * g, rtol=1e-5)


def test_grouped_score_with_caller_lse():
    """Only the column reduction, with the caller's [B, H * q_group, P]
    log-sum-exp (one per query head and proxy)."""
    B, H, g, L, D, P = 1, 3, 4, 1800, 128, 40
    w = custom("glse", B, H, L, D, P, dtype="bf16", data_seed=12)
    q, k, v = make_grouped_layer(w, g, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos)
    Fr, lse = proxy_scores_grouped(_f64(q), _f64(k), w.proxy_pos, prob.c.sm_scale, g)
    F = nacl.score(prob, q, k, nacl.workspace(prob), lse=torch.from_numpy(lse.astype(np.float32)).cuda())
    torch.cuda.synchronize()
    check_scores(F.cpu().numpy(), Fr, "grouped caller lse")


def test_grouped_eviction_matches_oracle():
    """32 query heads on 8 K/V heads at 4k tokens: scores, keep sets (per K/V
    head, Philox streams per K/V head) and compacted rows against the oracle."""
    B, H, g, L, D, P = 2, 8, 4, 4096, 128, 64
    w = custom("gevict", B, H, L, D, P, dtype="bf16", data_seed=33)
    q, k, v = make_grouped_layer(w, g, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos)
    F, keep, ko, vo = nacl.evict(prob, q, k, v, w.C, w.Cr, SAMPLE_SOFTMAX, 9, 4, ws=nacl.workspace(prob))
    torch.cuda.synchronize()
    Fr, _ = proxy_scores_grouped(_f64(q), _f64(k), w.proxy_pos, prob.c.sm_scale, g)
    check_scores(F.cpu().numpy(), Fr, "grouped evict F")
    kg = keep.cpu().numpy()
    check_keep_valid(kg, L, w.C, w.proxy_pos)
    n = 0
    for b in range(B):
        for h in range(H):
            Fr32 = Fr[b, h].astype(np.float32)
            ref = select_head(Fr32, w.proxy_pos, w.n_protect, w.C, w.Cr, SAMPLE_SOFTMAX, 9, 4, b, h)
            n += check_keep_near(kg[b, h], ref, Fr32, w.Cr, f"grouped keep b={b} h={h}")
            check_rows_for_common(kg[b, h], ko[b, h].cpu().view(torch.int16).numpy(), ref["keep"],
                                  k[b, h].cpu().view(torch.int16).numpy()[ref["keep"]], f"grouped K' b={b} h={h}")
            check_rows_for_common(kg[b, h], vo[b, h].cpu().view(torch.int16).numpy(), ref["keep"],
                                  v[b, h].cpu().view(torch.int16).numpy()[ref["keep"]], f"grouped V' b={b} h={h}")
    print(f"  grouped eviction: {n} near-tie differences", file=sys.stderr, flush=True)
