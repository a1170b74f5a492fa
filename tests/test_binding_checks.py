"""The Python binding refuses tensors that the kernels would address wrongly (host memory,
wrong shape, dtype or strides) before anything reaches the GPU, so these run on the CPU."""

import pytest
import torch

nacl = pytest.importorskip("paper_2408_03675_amd.nacl")


@pytest.fixture(scope="module")
def prob():
    nacl.load_library()
    return nacl.Problem(1, 2, 64, 64, "bf16", [60, 61, 62, 63])


def test_host_tensors_are_refused(prob):
    q = torch.zeros((1, 2, 64, 64), dtype=torch.bfloat16)
    ws = torch.zeros(16, dtype=torch.uint8)
    with pytest.raises(ValueError, match="on the GPU"):
        nacl.score(prob, q, q, ws)
    with pytest.raises(ValueError, match="on the GPU"):
        nacl.select(prob, torch.zeros((1, 2, 64)), 8, 2, ws=ws)
    with pytest.raises(ValueError, match="on the GPU"):
        nacl.compact(prob, q, q, torch.zeros((1, 2, 8), dtype=torch.int32))
    with pytest.raises(ValueError, match="on the GPU"):
        nacl.evict(prob, q, q, q, 8, 2, ws=ws)


def test_device_copy_of_proxy_positions_is_checked():
    with pytest.raises(ValueError, match="proxy_pos_dev"):
        nacl.Problem(1, 1, 16, 64, "bf16", [15], proxy_pos_dev=torch.tensor([15], dtype=torch.int64))
