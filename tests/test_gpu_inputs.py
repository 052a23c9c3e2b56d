"""The seeded input generator draws bit-identical values on the GPU and on the CPU (the oracle's inputs
are redrawn on the host), including the x4-scaled segment of the mixed batch and the normal's tails."""
import pytest
import torch

from paper_2608_01150_amd import workloads as W
from tests._gpu import HAVE_GPU

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="needs a GPU")]


@pytest.mark.parametrize("name,tensor", [("c2", W.TENSOR_V), ("c3", W.TENSOR_Q), ("c3", W.TENSOR_K), ("c4", W.TENSOR_DO)])
def test_device_draw_equals_cpu_draw(name, tensor):
    w = W.get(name)
    rows = 4000
    gpu = w.slice(tensor, 0, rows, device="cuda").cpu()
    cpu = w.slice(tensor, 0, rows)
    assert torch.equal(gpu, cpu)
    x = cpu.float()
    if not (name == "c3" and tensor in (W.TENSOR_Q, W.TENSOR_K)):   # c3's first rows are the x4 video
        assert abs(x.mean().item()) < 0.01 and abs(x.std().item() - 1) < 0.01
        assert x.abs().max().item() > 4.0       # a Gaussian tail, not a bounded stand-in
