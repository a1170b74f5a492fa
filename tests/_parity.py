"""Comparison rules between the GPU library and the CPU oracle.

Scores: |F_gpu - F_ref| <= 1e-3 * F_ref element-wise (fp32 accumulation
against float64), with an absolute floor of 1e-12 for scores near zero.

Keep sets: identical, except that every token in the symmetric difference
must sit at one of the oracle's two selection boundaries: its score within
1e-3 relative of the oracle's Cp-th best score, or its rank in the oracle's
random-key ordering within the band [Cr - n, Cr + n) where n is the size of
the difference.  Such near-ties can flip when fp32 scores differ in the last
bits; nothing else may.

Compaction: for every token kept by both sides, the GPU's row is bit-equal to
the oracle's row for that token.
"""

import numpy as np

F_RTOL = 1e-3
F_ATOL = 1e-12


def check_scores(F_gpu, F_ref, label=""):
    F_gpu = np.asarray(F_gpu, dtype=np.float64)
    F_ref = np.asarray(F_ref, dtype=np.float64)
    assert F_gpu.shape == F_ref.shape
    assert np.isfinite(F_gpu).all(), f"{label}: non-finite scores"
    err = np.abs(F_gpu - F_ref)
    bad = err > F_RTOL * np.abs(F_ref) + F_ATOL
    if bad.any():
        idx = np.argwhere(bad)[:5]
        raise AssertionError(f"{label}: {int(bad.sum())} scores off; first {idx.tolist()} "
                             f"gpu={F_gpu[tuple(idx[0])]} ref={F_ref[tuple(idx[0])]}")
    rel = (err / np.maximum(np.abs(F_ref), 1e-30)).max()
    return float(rel)


def check_keep_valid(keep, L, C, protected):
    keep = np.asarray(keep)
    assert keep.shape[-1] == C
    assert (np.diff(keep, axis=-1) > 0).all(), "keep_idx must be strictly ascending"
    if C:
        assert keep.min() >= 0 and keep.max() < L
    prot = set(int(x) for x in protected)
    for row in keep.reshape(-1, C):
        assert prot <= set(row.tolist())


def check_keep_near(keep_gpu, ref_head, F_ref32, Cr, label=""):
    """keep_gpu: 1-D GPU keep set of one head.  ref_head: the oracle's
    select_head dict for the same head.  F_ref32: oracle scores (fp32)."""
    g = set(int(x) for x in keep_gpu)
    r = set(int(x) for x in ref_head["keep"])
    diff = g ^ r
    if not diff:
        return 0
    n = len(diff)
    C = len(ref_head["keep"])
    assert n <= max(4, C // 500), f"{label}: {n} tokens differ out of {C}"
    F = np.asarray(F_ref32, dtype=np.float64)
    us = ref_head["u_score"]
    T1 = F[us].min() if len(us) else None
    key = ref_head["key"].astype(np.float64)
    taken = set(ref_head["protected"].tolist()) | set(us.tolist())
    R2 = np.array(sorted(set(range(len(F))) - taken), dtype=np.int64)
    order = R2[np.lexsort((R2, -key[R2]))]
    rank = {int(j): i for i, j in enumerate(order)}
    for j in diff:
        near_score = T1 is not None and abs(F[j] - T1) <= 1e-3 * abs(T1)
        near_random = j in rank and Cr - n <= rank[j] < Cr + n
        assert near_score or near_random, f"{label}: token {j} differs and is not a near-tie"
    return n


def check_rows_for_common(keep_gpu, rows_gpu, keep_ref, rows_ref, label=""):
    """Rows for tokens kept by both sides must be bit-identical."""
    kg = {int(j): c for c, j in enumerate(keep_gpu)}
    kr = {int(j): c for c, j in enumerate(keep_ref)}
    common = sorted(set(kg) & set(kr))
    a = np.ascontiguousarray(rows_gpu[[kg[j] for j in common]]).view(np.uint8)
    b = np.ascontiguousarray(rows_ref[[kr[j] for j in common]]).view(np.uint8)
    assert np.array_equal(a, b), f"{label}: compacted rows differ"
    return len(common)
