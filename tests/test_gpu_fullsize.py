"""GPU parity at the full workload sizes, through the same entry points and
launch configuration the benchmark times.

Every head is checked for properties that hold at any size (score mass per
head equals the proxy count, keep sets valid); sampled heads are checked
element by element against the CPU oracle (scores within 1e-3 relative,
keep sets equal up to near-ties, compacted rows bit-exact).
"""

import sys

import numpy as np
import pytest
import torch

from oracle import SAMPLE_SOFTMAX, proxy_scores, select_head
from synth import WORKLOADS, make_layer, sweep_workloads
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


def _check_heads(w, layer, q, k, v, F, keep, ko, vo, heads, label):
    """Element-wise parity of sampled heads against the oracle."""
    view = torch.int16 if w.dtype == "bf16" else torch.int32
    n_diff = 0
    for (b, h) in heads:
        Fr, _ = proxy_scores(_f64(q[b:b + 1, h:h + 1]), _f64(k[b:b + 1, h:h + 1]), w.proxy_pos, w.scale)
        check_scores(F[b, h].cpu().numpy(), Fr[0, 0], f"{label} F b={b} h={h}")
        Fr32 = Fr[0, 0].astype(np.float32)
        ref = select_head(Fr32, w.proxy_pos, w.n_protect, w.C, w.Cr, SAMPLE_SOFTMAX, w.rng_seed, layer, b, h)
        kg = keep[b, h].cpu().numpy()
        n_diff += check_keep_near(kg, ref, Fr32, w.Cr, f"{label} keep b={b} h={h}")
        kbits = k[b, h].cpu().view(view).numpy()
        vbits = v[b, h].cpu().view(view).numpy()
        check_rows_for_common(kg, ko[b, h].cpu().view(view).numpy(), ref["keep"], kbits[ref["keep"]],
                              f"{label} K' b={b} h={h}")
        check_rows_for_common(kg, vo[b, h].cpu().view(view).numpy(), ref["keep"], vbits[ref["keep"]],
                              f"{label} V' b={b} h={h}")
    return n_diff


def _properties(w, F, keep):
    Fs = F.double().sum(-1).cpu().numpy()
    np.testing.assert_allclose(Fs, w.P, rtol=1e-4)
    check_keep_valid(keep.cpu().numpy(), w.L, w.C, w.proxy_pos[w.P - w.n_protect:])


def _evict(w, layer):
    q, k, v = make_layer(w, layer, device="cuda")
    pos_dev = torch.tensor(w.proxy_pos, dtype=torch.int32, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos, n_protect=w.n_protect, sm_scale=w.scale,
                                     proxy_pos_dev=pos_dev)
    ws = nacl.workspace(prob)
    F, keep, ko, vo = nacl.evict(prob, q, k, v, w.C, w.Cr, SAMPLE_SOFTMAX, w.rng_seed, layer, ws=ws)
    torch.cuda.synchronize()
    status = int(ws[4:8].view(torch.int32).item())
    assert status == 0, "score kernel wait hit its spin limit"
    return q, k, v, F, keep, ko, vo


@pytest.mark.parametrize("layer", [0, 31])
def test_prefill_32k_layer(layer):
    """Batch 4 x 32 heads x 32768 tokens, 128 proxies, 20 % budget with half
    of it random: all heads' properties, six heads against the oracle."""
    w = WORKLOADS["prefill_32k"]
    _say("prefill_32k layer", layer)
    q, k, v, F, keep, ko, vo = _evict(w, layer)
    _properties(w, F, keep)
    heads = [(0, 0), (1, 7), (2, 19), (3, 31), (0, 16), (3, 3)]
    n = _check_heads(w, layer, q, k, v, F, keep, ko, vo, heads, f"32k L{layer}")
    _say(f"  {len(heads)} heads compared, {n} near-tie differences")


def test_sweep_16k_all_budgets():
    """Batch 8 x 32 heads x 16384 tokens; budgets 10/20/50 % with random
    shares 0/25/50 %: scores once, then selection and compaction per budget."""
    base = WORKLOADS["sweep_16k"]
    q, k, v = make_layer(base, 0, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, base.proxy_pos, sm_scale=base.scale)
    ws = nacl.workspace(prob)
    F = nacl.score(prob, q, k, ws)
    torch.cuda.synchronize()
    np.testing.assert_allclose(F.double().sum(-1).cpu().numpy(), base.P, rtol=1e-4)
    heads = [(0, 0), (5, 21), (7, 31)]
    refs = {}
    for (b, h) in heads:
        Fr, _ = proxy_scores(_f64(q[b:b + 1, h:h + 1]), _f64(k[b:b + 1, h:h + 1]), base.proxy_pos, base.scale)
        check_scores(F[b, h].cpu().numpy(), Fr[0, 0], f"16k F b={b} h={h}")
        refs[(b, h)] = Fr[0, 0].astype(np.float32)
    view = torch.int16
    for w in sweep_workloads():
        _say("sweep", w.name, "C", w.C, "Cr", w.Cr)
        keep = nacl.select(prob, F, w.C, w.Cr, SAMPLE_SOFTMAX, w.rng_seed, 0, ws=ws)
        ko, vo = nacl.compact(prob, k, v, keep)
        torch.cuda.synchronize()
        check_keep_valid(keep.cpu().numpy(), w.L, w.C, w.proxy_pos[w.P - w.n_protect:])
        for (b, h) in heads:
            ref = select_head(refs[(b, h)], w.proxy_pos, w.n_protect, w.C, w.Cr, SAMPLE_SOFTMAX, w.rng_seed,
                              0, b, h)
            kg = keep[b, h].cpu().numpy()
            check_keep_near(kg, ref, refs[(b, h)], w.Cr, f"{w.name} b={b} h={h}")
            kbits = k[b, h].cpu().view(view).numpy()
            check_rows_for_common(kg, ko[b, h].cpu().view(view).numpy(), ref["keep"], kbits[ref["keep"]],
                                  f"{w.name} K' b={b} h={h}")


def test_long_128k():
    """One sequence x 32 heads x 131072 tokens, 512 proxies (four proxy
    groups), heads too long for LDS-resident selection."""
    w = WORKLOADS["long_128k"]
    q, k, v, F, keep, ko, vo = _evict(w, 0)
    _properties(w, F, keep)
    n = _check_heads(w, 0, q, k, v, F, keep, ko, vo, [(0, 0), (0, 29)], "128k")
    _say(f"  128k: {n} near-tie differences")


def test_h2o_4k():
    """The H2O case of the scoring rule: batch 4 x 32 heads x 4096 tokens, every token
    a proxy (eight groups of 512 rows through the wide kernel, the API's proxy limit),
    none protected, the budget filled by score alone."""
    w = WORKLOADS["h2o_4k"]
    q, k, v, F, keep, ko, vo = _evict(w, 0)
    _properties(w, F, keep)
    n = _check_heads(w, 0, q, k, v, F, keep, ko, vo, [(0, 0), (3, 17)], "h2o_4k")
    _say(f"  h2o_4k: {n} near-tie differences")


def test_size_limits():
    """The API's limits: P = 4096 proxies (every token of a 4096-token head, the H2O-like
    case; the wide kernel over eight groups of 512), and one head of L = 2^19 tokens
    through the whole eviction (the selection kernel that re-reads keys from memory)."""
    from synth import custom
    w = custom("p_limit", 1, 1, 4096, 128, 4096, dtype="bf16", data_seed=21)
    q, k, v = make_layer(w, 0, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos, sm_scale=w.scale)
    F = nacl.score(prob, q, k, nacl.workspace(prob))
    torch.cuda.synchronize()
    Fr, _ = proxy_scores(_f64(q), _f64(k), w.proxy_pos, w.scale)
    check_scores(F.cpu().numpy(), Fr, "P = 4096")

    w = custom("l_limit", 1, 1, 1 << 19, 128, 16, dtype="bf16", inject=True, data_seed=22)
    _say("L = 2^19 eviction")
    q, k, v, F, keep, ko, vo = _evict(w, 0)
    _properties(w, F, keep)
    n = _check_heads(w, 0, q, k, v, F, keep, ko, vo, [(0, 0)], "L = 2^19")
    _say(f"  1 head compared, {n} near-tie differences")
