"""Reference samplers used to pin the oracle's random eviction (Section 5.2).

TEST INFRASTRUCTURE ONLY (see the oracle package docstring).

Section 5.2 draws |S_random| = Cr tokens from P_prompt = Softmax(F).  Read as
sampling without replacement, the probability of an ordered draw
(j_1, ..., j_k) is the Plackett-Luce product

    prod_t  w_{j_t} / (W - w_{j_1} - ... - w_{j_{t-1}}),   W = sum of w.

These helpers compute that law exactly for tiny inputs and draw from it
literally, one token at a time, so the Gumbel-top-k construction the oracle
uses can be checked against the definition.
"""

import itertools

import numpy as np


def set_probabilities(weights, k):
    """Exact probability of every k-subset under successive sampling without
    replacement.  Returns {tuple(sorted subset): probability}."""
    w = np.asarray(weights, dtype=np.float64)
    n = w.shape[0]
    total = w.sum()
    out = {}
    for perm in itertools.permutations(range(n), k):
        p = 1.0
        rest = total
        for j in perm:
            p *= w[j] / rest
            rest -= w[j]
        key = tuple(sorted(perm))
        out[key] = out.get(key, 0.0) + p
    return out


def sequential_sample(weights, k, rng):
    """Draw k distinct indices one at a time, each from the renormalised
    remaining weights (the literal reading of Section 5.2)."""
    w = np.asarray(weights, dtype=np.float64).copy()
    chosen = []
    for _ in range(k):
        p = w / w.sum()
        j = int(rng.choice(w.shape[0], p=p))
        chosen.append(j)
        w[j] = 0.0
    return tuple(sorted(chosen))
