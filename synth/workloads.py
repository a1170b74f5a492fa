"""Seeded synthetic workloads for the eviction step (shared by tests, smoke
check and benchmark).

This module only builds inputs: shapes, budgets as integer counts, and seeded
random Q/K/V.  It holds none of the eviction arithmetic, so both the GPU
library's callers and the CPU oracle can take their inputs from here.

The shapes follow the paper's workloads: LLaMA2-7B attention (32 layers x 32
heads x head_dim 128; Section 1 and Section 6.4), batch 4 at 32k tokens
(Section 1), LongBench-length prompts of about 4k tokens (Section 6.1) and the
128k-token run of Appendix A.7.  No model weights or datasets exist here; the
Q/K/V tensors are Gaussian stand-ins with injected attention sinks and heavy
hitters so that the scores have the skew real attention shows (Section 4).
"""

from dataclasses import dataclass, field
from fractions import Fraction
import math

import torch


@dataclass(frozen=True)
class Workload:
    """One eviction problem family.  Budgets are fractions of L; counts are
    derived with exact rational arithmetic:
        C  = floor(keep_frac * L)
        Cr = floor(random_share * C)
        n_protect = P (every proxy is kept; Section 5.1), unless `protect`
                    says otherwise (0 for the H2O case: every token a proxy)
        Cp = C - n_protect - Cr
    """
    name: str
    layers: int
    B: int
    H: int
    L: int
    D: int
    dtype: str                     # "f32" or "bf16"
    P: int
    keep_frac: Fraction
    random_share: Fraction
    inject: bool                   # attention-sink + heavy-hitter keys
    hh_frac: Fraction = Fraction(1, 100)
    data_seed: int = 0
    rng_seed: int = 0              # Philox seed of the random eviction
    sm_scale: float = field(default=0.0)
    protect: int = -1              # protected proxies; -1: all of them

    @property
    def scale(self):
        return self.sm_scale if self.sm_scale else 1.0 / math.sqrt(self.D)

    @property
    def C(self):
        return math.floor(self.keep_frac * self.L)

    @property
    def Cr(self):
        return math.floor(self.random_share * self.C)

    @property
    def n_protect(self):
        return self.P if self.protect < 0 else self.protect

    @property
    def Cp(self):
        return self.C - self.n_protect - self.Cr

    @property
    def proxy_pos(self):
        """Proxy tokens at the end of the prompt, where the question sits
        (Section 5.1 and Appendix A.3)."""
        return list(range(self.L - self.P, self.L))

    def with_budget(self, keep_frac, random_share):
        d = dict(self.__dict__)
        d["keep_frac"] = Fraction(keep_frac)
        d["random_share"] = Fraction(random_share)
        d["name"] = f"{self.name}_f{float(keep_frac):g}_r{float(random_share):g}"
        return Workload(**d)

    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16


# Hyperparameter table of Appendix A.6, 20 % row: random eviction takes 12 of
# the 20 points, a random share of 3/5.
PAPER_RANDOM_SHARE_20 = Fraction(3, 5)

WORKLOADS = {
    # 1 layer, one sequence, 4 heads of 64 in fp32: small enough for the oracle.
    "small_f32": Workload("small_f32", 1, 1, 4, 2048, 64, "f32", 32,
                          Fraction(1, 5), PAPER_RANDOM_SHARE_20, False,
                          data_seed=1, sm_scale=0.125),
    # LLaMA2-7B layer shape at LongBench length.
    "longbench_4k": Workload("longbench_4k", 1, 1, 32, 4096, 128, "bf16", 64,
                             Fraction(1, 5), PAPER_RANDOM_SHARE_20, True,
                             data_seed=2),
    # All 32 layers, batch 4 at 32k tokens: the headline workload.
    "prefill_32k": Workload("prefill_32k", 32, 4, 32, 32768, 128, "bf16", 128,
                            Fraction(1, 5), Fraction(1, 2), True, data_seed=3),
    # Batch 8 at 16k; the budget/random-share sweep derives from it.
    "sweep_16k": Workload("sweep_16k", 1, 8, 32, 16384, 128, "bf16", 128,
                          Fraction(1, 5), Fraction(0), False, data_seed=4),
    # One sequence at 128k tokens (Appendix A.7's length).
    "long_128k": Workload("long_128k", 1, 1, 32, 131072, 128, "bf16", 512,
                          Fraction(1, 5), PAPER_RANDOM_SHARE_20, True,
                          hh_frac=Fraction(1, 1000), data_seed=5),
    # The H2O special case of the scoring rule (Section 5.1): every token a
    # proxy, none protected, the budget filled by score alone.  A dense,
    # MFMA-bound column sum over the whole causal attention matrix.
    "h2o_4k": Workload("h2o_4k", 1, 4, 32, 4096, 128, "bf16", 4096,
                       Fraction(1, 5), Fraction(0), True, data_seed=6, protect=0),
}

SWEEP_KEEP = (Fraction(1, 10), Fraction(1, 5), Fraction(1, 2))
SWEEP_RANDOM = (Fraction(0), Fraction(1, 4), Fraction(1, 2))


def sweep_workloads():
    base = WORKLOADS["sweep_16k"]
    return [base.with_budget(f, r) for f in SWEEP_KEEP for r in SWEEP_RANDOM]


def custom(name, B, H, L, D, P, dtype="bf16", keep_frac=Fraction(1, 5),
           random_share=PAPER_RANDOM_SHARE_20, inject=False, data_seed=0,
           rng_seed=0, sm_scale=0.0, hh_frac=Fraction(1, 100)):
    return Workload(name, 1, B, H, L, D, dtype, P, Fraction(keep_frac),
                    Fraction(random_share), inject, hh_frac, data_seed,
                    rng_seed, sm_scale)


def make_layer(w, layer=0, device="cpu"):
    """Seeded Q, K, V [B, H, L, D] for one layer of workload w.

    Values are N(0, 1) drawn in fp32 from a torch.Generator seeded with
    data_seed + 1000 * layer, then (if w.inject) attention-sink and
    heavy-hitter keys are added, then the tensors are rounded to w.dtype
    (round-to-nearest-even for bf16).

    Injection, per (b, h): u = normalised mean of the head's proxy queries;
    K[j] += alpha * sqrt(D) * u, which raises the logit of a query q by
    alpha * <q, u> at scale 1/sqrt(D).  alpha = 4 for the first four keys
    (attention sinks) and alpha = 2 for hh_frac of the keys drawn without
    replacement from [4, L - P) (heavy hitters).
    """
    gen = torch.Generator(device=device)
    gen.manual_seed(int(w.data_seed) + 1000 * int(layer))
    shape = (w.B, w.H, w.L, w.D)
    q = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
    k = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
    v = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
    if w.inject:
        pos = torch.tensor(w.proxy_pos, device=device, dtype=torch.long)
        u = q.index_select(2, pos).mean(dim=2)                     # [B, H, D]
        u = u / u.norm(dim=-1, keepdim=True).clamp_min(1e-12)
        push = math.sqrt(w.D) * u
        n_sink = min(4, w.L)
        k[:, :, :n_sink, :] += 4.0 * push[:, :, None, :]
        span = w.L - w.P - 4
        n_hh = math.floor(w.hh_frac * w.L)
        if span > 0 and n_hh > 0:
            n_hh = min(n_hh, span)
            r = torch.rand((w.B, w.H, span), generator=gen, device=device)
            hh = r.argsort(dim=-1)[..., :n_hh] + 4                  # [B, H, n_hh]
            add = (2.0 * push)[:, :, None, :].expand(w.B, w.H, n_hh, w.D)
            k.scatter_add_(2, hh[..., None].expand(w.B, w.H, n_hh, w.D), add)
    dt = w.torch_dtype()
    return q.to(dt), k.to(dt), v.to(dt)


def make_grouped_layer(w, q_group, layer=0, device="cpu"):
    """Q [B, H * q_group, L, D] and K, V [B, H, L, D] for grouped-query
    attention (several query heads per K/V head): N(0, 1) drawn in fp32 from
    a torch.Generator seeded with data_seed + 1000 * layer (Q first, then K,
    then V), rounded to w.dtype; no injection."""
    gen = torch.Generator(device=device)
    gen.manual_seed(int(w.data_seed) + 1000 * int(layer))
    q = torch.randn((w.B, w.H * q_group, w.L, w.D), generator=gen, device=device, dtype=torch.float32)
    k = torch.randn((w.B, w.H, w.L, w.D), generator=gen, device=device, dtype=torch.float32)
    v = torch.randn((w.B, w.H, w.L, w.D), generator=gen, device=device, dtype=torch.float32)
    dt = w.torch_dtype()
    return q.to(dt), k.to(dt), v.to(dt)


def alg_bytes(w):
    """Algorithmic HBM bytes of one layer, per stage (inputs read once,
    outputs written once).  Used for roofline fractions."""
    elt = 4 if w.dtype == "f32" else 2
    bh = w.B * w.H
    score = bh * (w.L * w.D * elt + w.P * w.D * elt + 4 * w.L)
    select = bh * (4 * w.L + 4 * w.C)
    compact = bh * (2 * 2 * w.C * w.D * elt + 4 * w.C)
    return {"score": score, "select": select, "compact": compact}


def alg_flops(w):
    """One Q_P K^T contraction per (b, h): 2 * P_eff * D flops per visible
    (proxy, key) pair, with the causal mask's visible-pair count."""
    pairs = sum(p + 1 for p in w.proxy_pos)
    return 2 * w.D * pairs * w.B * w.H
