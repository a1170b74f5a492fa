"""Plain CPU oracle of NaCl's one-shot encoding-phase KV-cache eviction.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code with
the GPU library and must never be used as a fallback for it.

Paper: Chen et al., "NaCl: A General and Effective KV Cache Eviction Framework
for LLMs at Inference Time" (arXiv 2408.03675).  Every function cites the
passage it follows.  Arithmetic is float64 (inputs in bf16 or fp32 convert to
float64 exactly); integer decisions are taken in float32, the precision the GPU
library decides in, so both sides rank identical values.

Per (layer l, batch row b, head h) the step is:

  1. score (Section 5.1, equation for F_score; Algorithm 1, encoding phase):
       A[i, j] = s * <Q[p_i], K[j]>  for j <= p_i (causal), s = sm_scale
       F[j]    = sum_i softmax_j(A[i, :])[j]
  2. u_score (Section 5.1, the argmax equation): the Cp tokens of
       R = [0, L) minus the protected proxies with the largest F, ties to the
       lower index, together with the protected proxies.
  3. u_random (Section 5.2): Cr tokens sampled without replacement from the
       remaining candidates with probabilities Softmax(F), drawn with the
       Gumbel-top-k construction from Philox4x32-10 uniforms.
  4. S = u_score | u_random, |S| = C, ascending (Algorithm 1).
  5. K', V' = K[S], V[S] (Section 3, encoding-phase cache update).

Readings of points where the paper is silent are listed in the design notes;
the ones that change arithmetic are restated at the function that uses them.
"""

import numpy as np

from .philox import token_words, open_unit

SAMPLE_SOFTMAX = 0       # weights proportional to exp(F): Softmax(F_score), Section 5.2
SAMPLE_PROPORTIONAL = 1  # weights proportional to F (variant, not the default)
SAMPLE_UNIFORM = 2       # equal weights (the ablation's uniform distribution)


def proxy_scores(Q, K, proxy_pos, sm_scale):
    """F_score of Section 5.1 for every (b, h): column sums of the proxy rows'
    causal softmax.

    Q, K: arrays [B, H, L, D] (any float dtype; converted to float64).
    proxy_pos: strictly increasing int positions p_1 < ... < p_P in [0, L).
    sm_scale: the logit scale s (the paper divides by sqrt(d); Algorithm 1).

    Reading: the attention matrix is causal (decoder-only model, and the
    FlashAttention-2 log-sum-exp the appendix reuses is causal), so proxy row i
    covers keys 0..p_i, itself included.

    Returns (F, lse): F float64 [B, H, L]; lse float64 [B, H, P] is the natural
    log-sum-exp of each proxy row's scaled logits (the quantity the appendix's
    reduce algorithm takes from FlashAttention-2).
    """
    Q = np.asarray(Q)
    K = np.asarray(K)
    pos = np.asarray(proxy_pos, dtype=np.int64)
    B, H, L, D = K.shape
    P = pos.shape[0]
    s = np.float64(sm_scale)
    keys = np.arange(L, dtype=np.int64)
    visible = keys[None, :] <= pos[:, None]              # [P, L] causal mask
    F = np.zeros((B, H, L), dtype=np.float64)
    lse = np.zeros((B, H, P), dtype=np.float64)
    for b in range(B):
        for h in range(H):
            Qp = Q[b, h, pos, :].astype(np.float64)       # Q_P: the proxy rows
            Kh = K[b, h].astype(np.float64)
            A = s * (Qp @ Kh.T)                           # [P, L] logits
            A = np.where(visible, A, -np.inf)
            m = A.max(axis=1, keepdims=True)
            row_lse = m + np.log(np.exp(A - m).sum(axis=1, keepdims=True))
            pi = np.exp(A - row_lse)                      # softmax rows; 0 where masked
            F[b, h] = pi.sum(axis=0)                      # sum over proxy rows
            lse[b, h] = row_lse[:, 0]
    return F, lse


def proxy_scores_grouped(Q, K, proxy_pos, sm_scale, q_group):
    """F_score (Section 5.1) when several query heads share one K/V head
    (grouped-query attention; the paper's LLaMA2-7B has one query head per
    K/V head, so this is a reading for models that group them).

    Reading: the attention rows that look at K/V head h are those of its
    q_group query heads h * q_group .. h * q_group + q_group - 1, so K/V head h
    is scored by the proxy rows of all of them: F[b, h] is the sum over the
    group of each query head's F_score against the shared keys, and its score
    mass is P * q_group.

    Q: [B, H * q_group, L, D]; K: [B, H, L, D].  Returns (F [B, H, L],
    lse [B, H * q_group, P]), float64.
    """
    Q = np.asarray(Q)
    K = np.asarray(K)
    B, H, L, D = K.shape
    g = int(q_group)
    if Q.shape[1] != H * g:
        raise ValueError("Q must have H * q_group heads")
    F = np.zeros((B, H, L), dtype=np.float64)
    lse = np.zeros((B, H * g, len(proxy_pos)), dtype=np.float64)
    for h in range(H):
        for e in range(g):
            hq = h * g + e
            Fe, le = proxy_scores(Q[:, hq:hq + 1], K[:, h:h + 1], proxy_pos, sm_scale)
            F[:, h] += Fe[:, 0]
            lse[:, hq] = le[:, 0]
    return F, lse


def causal_attention(Q, K, V, sm_scale, q_group=1, rows=None):
    """The prefill's causal attention and its per-row log-sum-exp: the
    forward pass whose log-sum-exp the appendix on FlashAttention-2
    (Appendix A.7, the paragraph before Algorithm 2) hands to the score so
    that only the column reduction remains.

    For query head hq (K/V head hq // q_group, the grouping of
    proxy_scores_grouped) and row i:
        A[i, j] = s * <Q[i], K[j]>, j <= i (causal)
        lse[i]  = log sum_{j <= i} exp(A[i, j])
        O[i]    = sum_{j <= i} exp(A[i, j] - lse[i]) * V[j]

    Q: [B, H * q_group, L, D]; K, V: [B, H, L, D].  rows: optional int array
    of query rows (all rows when None).  Returns (O [B, H * q_group, n, D],
    lse [B, H * q_group, n]) in float64, n = number of rows.
    """
    Q = np.asarray(Q)
    K = np.asarray(K)
    V = np.asarray(V)
    B, H, L, D = K.shape
    g = int(q_group) if q_group and q_group > 1 else 1
    if Q.shape[1] != H * g:
        raise ValueError("Q must have H * q_group heads")
    r = np.arange(L, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    s = np.float64(sm_scale)
    visible = np.arange(L, dtype=np.int64)[None, :] <= r[:, None]   # [n, L]
    O = np.zeros((B, H * g, r.shape[0], D), dtype=np.float64)
    lse = np.zeros((B, H * g, r.shape[0]), dtype=np.float64)
    for b in range(B):
        for hq in range(H * g):
            h = hq // g
            Kh = K[b, h].astype(np.float64)
            Vh = V[b, h].astype(np.float64)
            A = s * (Q[b, hq, r, :].astype(np.float64) @ Kh.T)    # [n, L]
            A = np.where(visible, A, -np.inf)
            m = A.max(axis=1, keepdims=True)
            row_lse = m + np.log(np.exp(A - m).sum(axis=1, keepdims=True))
            O[b, hq] = np.exp(A - row_lse) @ Vh
            lse[b, hq] = row_lse[:, 0]
    return O, lse


def protected_set(proxy_pos, n_protect):
    """Pi: the proxy tokens kept by default (Section 5.1: proxies are retained).

    Reading of the hyperparameter table (Appendix A.6, "Protect Proxy"): only
    the last n_protect proxies are force-kept; the default n_protect = P keeps
    them all, as the main text says.
    """
    pos = np.asarray(proxy_pos, dtype=np.int64)
    P = pos.shape[0]
    if not 0 <= n_protect <= P:
        raise ValueError("n_protect out of range")
    return pos[P - n_protect:]


def budget_split(C, Cr, n_protect):
    """C = |Pi| + Cp + Cr (Algorithm 1 states C = Cp + Cr; the hyperparameter
    table's columns add up to the budget, so protected proxies count inside
    it).  Returns Cp."""
    Cp = C - n_protect - Cr
    if Cr < 0 or Cp < 0:
        raise ValueError("budget too small for the protected proxies and Cr")
    return Cp


def top_k_lower_index(values, candidates, k):
    """The k candidates with the largest value; equal values go to the lower
    index (a reading: the paper does not order ties).  Returns an int64 array
    of indices in selection order."""
    cand = np.asarray(candidates, dtype=np.int64)
    v = np.asarray(values)[cand]
    order = np.lexsort((cand, -v.astype(np.float64)))
    return cand[order[:k]]


def gumbel_keys(F32, words, sampling):
    """Perturbed keys whose top-Cr is a sample without replacement (Section 5.2).

    Gumbel-top-k (Vieira 2014; Kool, van Hoof and Welling 2019): with
    g_j = -ln(-ln u_j), u_j uniform on (0, 1), the Cr largest of log w_j + g_j
    are distributed as Cr successive draws without replacement with
    probabilities proportional to w_j.  For Softmax(F) the log-weight is F
    itself.

    Precision: u and g are binary64; the key is the binary64 sum rounded once
    to binary32, and ranking happens on binary32 keys.
    """
    u = open_unit(words)
    g = -np.log(-np.log(u))
    F64 = np.asarray(F32, dtype=np.float32).astype(np.float64)
    if sampling == SAMPLE_SOFTMAX:
        key = F64 + g
    elif sampling == SAMPLE_PROPORTIONAL:
        with np.errstate(divide="ignore"):
            key = np.log(F64) + g
    elif sampling == SAMPLE_UNIFORM:
        key = g
    else:
        raise ValueError("unknown sampling mode")
    return key.astype(np.float32)


def select_head(F32, proxy_pos, n_protect, C, Cr, sampling, seed, layer, b, h):
    """Keep set S of one head (Algorithm 1, encoding phase).

    F32: float32 scores of one head, length L.  Returns a dict with the sorted
    keep indices and the three parts (protected, u_score, u_random).
    """
    F32 = np.asarray(F32, dtype=np.float32)
    L = F32.shape[0]
    if not 0 <= C <= L:
        raise ValueError("budget C must lie in [0, L]")
    Pi = protected_set(proxy_pos, n_protect)
    Cp = budget_split(C, Cr, n_protect)
    in_pi = np.zeros(L, dtype=bool)
    in_pi[Pi] = True
    R = np.flatnonzero(~in_pi)                            # R = x_prompt minus proxies
    u_score = top_k_lower_index(F32, R, Cp)               # top-Cp of F over R
    taken = in_pi.copy()
    taken[u_score] = True
    R2 = np.flatnonzero(~taken)                           # candidates left for sampling
    words = token_words(seed, layer, b, h, L)
    key = gumbel_keys(F32, words, sampling)
    u_random = top_k_lower_index(key, R2, Cr)
    keep = np.sort(np.concatenate([Pi, u_score, u_random]))
    return {"keep": keep, "protected": Pi, "u_score": np.sort(u_score),
            "u_random": np.sort(u_random), "key": key}


def select(F32, proxy_pos, n_protect, C, Cr, sampling, seed, layer):
    """keep_idx [B, H, C] int32, ascending per head (Algorithm 1)."""
    F32 = np.asarray(F32, dtype=np.float32)
    B, H, L = F32.shape
    out = np.zeros((B, H, C), dtype=np.int32)
    for b in range(B):
        for h in range(H):
            out[b, h] = select_head(F32[b, h], proxy_pos, n_protect, C, Cr,
                                    sampling, seed, layer, b, h)["keep"]
    return out


def compact(K, V, keep_idx):
    """K0, V0 <- K_S, V_S (Section 3, encoding-phase eviction): the kept rows,
    in keep order, copied exactly."""
    K = np.asarray(K)
    V = np.asarray(V)
    idx = np.asarray(keep_idx, dtype=np.int64)
    B, H, C = idx.shape
    bi = np.arange(B)[:, None, None]
    hi = np.arange(H)[None, :, None]
    return K[bi, hi, idx], V[bi, hi, idx]


def slot_layout(keep, C):
    """Where the kept rows of one head sit after a generation-phase eviction
    that leaves kept rows in place (Section 3, "Generation Phase Eviction";
    the paper fixes which entries stay, not their order in the cache): a kept
    row below C keeps its slot; the kept rows at or past C go, in ascending
    order, to the slots below C whose rows were not kept, also taken in
    ascending order.  keep: the ascending keep set (C rows).  Returns slot_src
    with slot_src[c] = the row slot c holds afterwards."""
    keep = [int(r) for r in keep]
    assert len(keep) == C and keep == sorted(set(keep))
    staying = [r for r in keep if r < C]
    movers = [r for r in keep if r >= C]
    taken = set(staying)
    free = [c for c in range(C) if c not in taken]
    assert len(free) == len(movers)
    slot_src = list(range(C))
    for c, r in zip(free, movers):
        slot_src[c] = r
    return np.array(slot_src, dtype=np.int64)


def evict(Q, K, V, proxy_pos, n_protect, C, Cr, sampling, seed, layer, sm_scale):
    """The whole step for one layer: score, select, compact."""
    F, lse = proxy_scores(Q, K, proxy_pos, sm_scale)
    F32 = F.astype(np.float32)
    keep = select(F32, proxy_pos, n_protect, C, Cr, sampling, seed, layer)
    Kc, Vc = compact(K, V, keep)
    return {"F": F, "lse": lse, "keep_idx": keep, "k_out": Kc, "v_out": Vc}
