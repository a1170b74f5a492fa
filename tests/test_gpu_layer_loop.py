"""The benchmark's timed configuration: the layer loop (Algorithm 1, encoding
phase, layer after layer) on two alternating streams with one workspace
each, as bench.py runs it, on a reduced 32k workload (batch 1, 4 layers).
Every layer's scores, keep set and compacted K/V must equal, bit for bit,
those of a one-layer nacl_evict call on one stream, and one head per layer
must match the oracle."""

import sys

import numpy as np
import pytest
import torch

from oracle import SAMPLE_SOFTMAX, proxy_scores, select_head
from synth import WORKLOADS, make_layer
from tests._parity import check_keep_near, check_rows_for_common, check_scores

pytestmark = pytest.mark.gpu

nacl = pytest.importorskip("paper_2408_03675_amd.nacl")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nacl.load_library()


def test_layer_loop_matches_single_layer_calls():
    from dataclasses import replace
    from paper_2408_03675_amd.layer_loop import LayerLoop
    w = replace(WORKLOADS["prefill_32k"], B=1, layers=4, name="prefill_32k_b1")
    dev = torch.device("cuda:0")
    data = [make_layer(w, ell, device=dev) for ell in range(w.layers)]
    pos_dev = torch.tensor(w.proxy_pos, dtype=torch.int32, device=dev)
    q0, k0, v0 = data[0]
    prob = nacl.Problem.from_tensors(q0, k0, v0, w.proxy_pos, sm_scale=w.scale, proxy_pos_dev=pos_dev)
    loop = LayerLoop(prob, data, w.C, w.Cr, SAMPLE_SOFTMAX, w.rng_seed, streams=2, device=dev)
    for _ in range(2):   # twice, as warm-up and timed steps reuse the workspaces
        loop.run()
    torch.cuda.synchronize()
    assert loop.health() == 0
    ws = nacl.workspace(prob, dev)
    heads = [(0, 3), (0, 17), (0, 30), (0, 9)]
    for ell, (q, k, v) in enumerate(data):
        print(f"layer {ell}", file=sys.stderr, flush=True)
        ref = nacl.evict(prob, q, k, v, w.C, w.Cr, SAMPLE_SOFTMAX, w.rng_seed, ell, ws=ws)
        torch.cuda.synchronize()
        assert nacl.health(ws) == (0, 0)
        for a, b, name in zip(loop.outs[ell], ref, ("scores", "keep_idx", "k_out", "v_out")):
            ai = a.view(torch.int32) if a.dtype == torch.float32 else (a.view(torch.int16) if a.dtype == torch.bfloat16 else a)
            bi = b.view(torch.int32) if b.dtype == torch.float32 else (b.view(torch.int16) if b.dtype == torch.bfloat16 else b)
            assert torch.equal(ai, bi), f"layer {ell}: {name} differs from the one-layer call"
        bb, h = heads[ell]
        F, keep, ko, vo = loop.outs[ell]
        Fr, _ = proxy_scores(q[bb:bb + 1, h:h + 1].double().cpu().numpy(),
                             k[bb:bb + 1, h:h + 1].double().cpu().numpy(), w.proxy_pos, w.scale)
        check_scores(F[bb, h].cpu().numpy(), Fr[0, 0], f"layer {ell} F h={h}")
        Fr32 = Fr[0, 0].astype(np.float32)
        r = select_head(Fr32, w.proxy_pos, w.n_protect, w.C, w.Cr, SAMPLE_SOFTMAX, w.rng_seed, ell, bb, h)
        kg = keep[bb, h].cpu().numpy()
        check_keep_near(kg, r, Fr32, w.Cr, f"layer {ell} keep h={h}")
        kbits = k[bb, h].cpu().view(torch.int16).numpy()
        vbits = v[bb, h].cpu().view(torch.int16).numpy()
        check_rows_for_common(kg, ko[bb, h].cpu().view(torch.int16).numpy(), r["keep"], kbits[r["keep"]],
                              f"layer {ell} K'")
        check_rows_for_common(kg, vo[bb, h].cpu().view(torch.int16).numpy(), r["keep"], vbits[r["keep"]],
                              f"layer {ell} V'")
