"""Comparison rules between the GPU library and the CPU oracle.

Scores: |F_gpu - F_ref| <= 1e-3 * F_ref element-wise (fp32 accumulation
against float64), with an absolute floor of 1e-30: exponentials are taken in
binary32 on the GPU, so a term below binary32's normal range (about 1.2e-38)
may flush to zero; every term at or above 1e-30 must be kept.

Keep sets: identical, except for tokens whose membership a score error within
that tolerance can flip.  Each token in the symmetric difference must be one
of:
  - a score near-tie: |F[j] - T1| <= 1e-3 * (F[j] + T1) (+ floor), T1 the
    oracle's Cp-th best score over R (Section 5.1 argmax): two errors within
    the tolerance can swap such a token with the boundary one;
  - a random near-tie: its oracle Gumbel key within the shift that such score
    errors (plus one binary32 rounding of each key) can cause of the oracle's
    Cr-th key over R \\ u_score (Section 5.2);
  - a cascade of score near-ties: when u_score trades a token with the
    candidates of the random draw, the draw's boundary moves by one rank per
    traded token, so ranks within [Cr - a, Cr + a) of the oracle's random-key
    order are allowed, a being the number of trades the score tie band
    allows (its members inside u_score or outside it, whichever are fewer).
Nothing else may differ.

Compaction: for every token kept by both sides, the GPU's row is bit-equal to
the oracle's row for that token.
"""

import numpy as np

F_RTOL = 1e-3
F_ATOL = 1e-30

SAMPLE_SOFTMAX, SAMPLE_PROPORTIONAL, SAMPLE_UNIFORM = 0, 1, 2


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


def _key_shift(F, j, t, mode, key):
    """Largest change in key[j] - key[t] that score errors within the
    tolerance, and one binary32 rounding of each key, can cause."""
    ulp = 2.0 * np.spacing(np.float32(max(abs(float(key[j])), abs(float(key[t])))))
    if mode == SAMPLE_SOFTMAX:          # key = F + g
        return F_RTOL * (F[j] + F[t]) + 2 * F_ATOL + float(ulp)
    if mode == SAMPLE_PROPORTIONAL:     # key = ln F + g
        return 2.0 * np.log1p(F_RTOL) + float(ulp)
    return float(ulp)                   # uniform: g alone


def check_keep_near(keep_gpu, ref_head, F_ref32, Cr, label="", mode=SAMPLE_SOFTMAX):
    """keep_gpu: 1-D GPU keep set of one head.  ref_head: the oracle's
    select_head dict for the same head.  F_ref32: oracle scores (fp32).
    mode: the sampling distribution the keys were drawn for."""
    g = set(int(x) for x in keep_gpu)
    r = set(int(x) for x in ref_head["keep"])
    diff = g ^ r
    if not diff:
        return 0
    n = len(diff)
    C = len(ref_head["keep"])
    assert n <= max(4, C // 500), f"{label}: {n} tokens differ out of {C}"
    F = np.asarray(F_ref32, dtype=np.float64)
    L = len(F)
    prot = set(ref_head["protected"].tolist())
    us = ref_head["u_score"]
    R = np.array(sorted(set(range(L)) - prot), dtype=np.int64)
    T1 = None
    a = 0
    if len(us):
        T1 = F[us].min()
        near = np.abs(F[R] - T1) <= F_RTOL * (F[R] + T1) + F_ATOL
        inside = np.isin(R, us)
        a = int(min((near & inside).sum(), (near & ~inside).sum()))  # boundary trades possible
    key = ref_head["key"].astype(np.float64)
    R2 = np.array(sorted(set(R.tolist()) - set(us.tolist())), dtype=np.int64)
    order = R2[np.lexsort((R2, -key[R2]))]
    rank = {int(j): i for i, j in enumerate(order)}
    t_r = int(order[Cr - 1]) if 0 < Cr <= len(order) else None
    for j in diff:
        near_score = T1 is not None and abs(F[j] - T1) <= F_RTOL * (F[j] + T1) + F_ATOL
        near_key = t_r is not None and j in rank and \
            abs(key[j] - key[t_r]) <= _key_shift(F, j, t_r, mode, key)
        cascade = j in rank and Cr - a <= rank[j] < Cr + a
        assert near_score or near_key or cascade, \
            f"{label}: token {j} differs and is not a near-tie (rank {rank.get(j)}, Cr {Cr}, band {a})"
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
