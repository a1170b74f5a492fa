"""nacl_evict_noalloc (the entry point for callers that cannot allocate)
against nacl_evict with a caller workspace: calls in a row on the same
GPU, the second on a smaller problem and the third on a few-row one (the
built-in scratch keeps the previous call's contents), each compared bit for
bit with nacl_evict on the same inputs (the same kernels run, so scores, keep
sets and compacted rows are identical), plus one head against the oracle;
health words zero.  A problem whose workspace exceeds the built-in scratch
is refused."""

import numpy as np
import pytest
import torch

from oracle import SAMPLE_SOFTMAX, proxy_scores, select_head
from synth import custom, make_layer
from tests._parity import check_keep_near, check_scores

pytestmark = pytest.mark.gpu

nacl = pytest.importorskip("paper_2408_03675_amd.nacl")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nacl.load_library()


def _bits(t):
    return t.view(torch.int32) if t.dtype == torch.float32 else (t.view(torch.int16) if t.dtype == torch.bfloat16 else t)


def _case(w):
    q, k, v = make_layer(w, 0, device="cuda")
    pos_dev = torch.tensor(w.proxy_pos, dtype=torch.int32, device="cuda")
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos, sm_scale=w.scale, proxy_pos_dev=pos_dev)
    health = torch.full((2,), -1, dtype=torch.int32, device="cuda")
    got = nacl.evict_noalloc(prob, q, k, v, w.C, w.Cr, SAMPLE_SOFTMAX, 3, 1, health=health)
    ref = nacl.evict(prob, q, k, v, w.C, w.Cr, SAMPLE_SOFTMAX, 3, 1, ws=nacl.workspace(prob))
    torch.cuda.synchronize()
    assert health.tolist() == [0, 0]
    for a, b, name in zip(got, ref, ("scores", "keep_idx", "k_out", "v_out")):
        assert torch.equal(_bits(a), _bits(b)), f"{w.name}: {name} differs from nacl_evict"
    F, keep = got[0], got[1]
    Fr, _ = proxy_scores(q[:1, :1].double().cpu().numpy(), k[:1, :1].double().cpu().numpy(), w.proxy_pos, w.scale)
    check_scores(F[0, 0].cpu().numpy(), Fr[0, 0], f"{w.name} F")
    Fr32 = Fr[0, 0].astype(np.float32)
    r = select_head(Fr32, w.proxy_pos, w.n_protect, w.C, w.Cr, SAMPLE_SOFTMAX, 3, 1, 0, 0)
    check_keep_near(keep[0, 0].cpu().numpy(), r, Fr32, w.Cr, f"{w.name} keep")


def test_noalloc_matches_evict_twice_smaller_second():
    _case(custom("noalloc_big", 2, 8, 9000, 128, 128, dtype="bf16", inject=True, data_seed=71))
    _case(custom("noalloc_small", 1, 3, 2100, 64, 40, dtype="f32", data_seed=72))
    # a third call: two proxies, the few-row score path (logits in the scratch)
    _case(custom("noalloc_rows", 2, 4, 3001, 128, 2, dtype="bf16", data_seed=73))


def test_noalloc_refuses_oversized_problems():
    L = 1 << 19
    prob = nacl.Problem(16, 32, L, 128, "bf16", list(range(L - 128, L)))
    assert nacl.workspace_bytes(prob) > nacl.NOALLOC_WORKSPACE_MAX
    lib = nacl.load_library()
    fake = torch.empty(16, device="cuda")
    st = lib.nacl_evict_noalloc(prob.ref(), fake.data_ptr(), fake.data_ptr(), fake.data_ptr(), 10, 0, 0, 0, 0,
                                fake.data_ptr(), fake.data_ptr(), fake.data_ptr(), fake.data_ptr(), None, None)
    assert st == nacl.NACL_ERR_UNSUPPORTED
    assert b"scratch" in lib.nacl_last_error_detail()
