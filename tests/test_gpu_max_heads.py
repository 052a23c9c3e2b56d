"""The largest head count the library accepts (ZL_MAX_HEADS = 16384, d = 128).
Consecutive tokens of Q, K, V are then 4 MiB apart, and a 64-row tile load
spans 252 MiB of the 32-bit byte offsets the kernels use within a tile.  A
packed batch runs the forward, the merge and the backward over all heads: a
WHOLE segment of 1100 rows, which puts every later segment more than 4 GiB
into the tensors (4.3 GiB: 64-bit bases beside the 32-bit in-tile offsets),
then a WHOLE segment of 70 rows (a full and a ragged tile) and a SHARD of 40
rows against blocks of 50 and 30 keys.  Sampled heads (both ends and seeded
others) are checked against the oracle run on those heads alone: attention
never mixes heads, so that is the full oracle restricted to them."""
import numpy as np
import pytest
import torch

import oracle
from tests import _descs
from tests._gpu import HAVE_GPU, api, to64
from tests.test_gpu_parity import LSE_TOL, O_TOL, _check_bwd

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="needs a GPU")]

H, HD = 16384, 128


@pytest.fixture
def release_cache():
    yield
    torch.cuda.empty_cache()  # about 62 GB of tensors; later tests in the process need none of it


def test_max_heads_forward_merge_backward(release_cache):
    d = _descs.desc(cu_q=(0, 1100, 1170, 1210), kind=(0, 0, 1), kv_first=(0, 1, 2), kv_count=(1, 1, 2),
                    cu_k=(0, 1100, 1170, 1220, 1250), block_index=(0, 0, 1, 0), num_slots=2,
                    q_offset=(0, 0, 0), k_offset=(0, 0, 0, 50))
    tq, tk = 1210, 1250
    assert 1100 * H * HD * 2 > 1 << 32
    desc = api.SegDesc.of(d)
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(16384)
    q, k, v, do = (torch.randn((n, H, HD), generator=g, device=dev, dtype=torch.bfloat16)
                   for n in (tq, tk, tk, tq))
    scale = HD ** -0.5
    print(f"max heads: H={H} d={HD} Tq={tq} Tk={tk}", flush=True)

    out, lse, o_part, lse_part = api.attn_fwd(desc, q, k, v, scale)
    torch.cuda.synchronize()
    o_part_shard = o_part[:, 1170:].clone()  # the shard's partials, before the merge
    lse_part_shard = lse_part[:, 1170:].clone()
    api.lse_merge(desc, o_part, lse_part, out, lse)
    dq, dk, dv = api.attn_bwd(desc, q, k, v, out, lse, do, scale)
    torch.cuda.synchronize()

    rng = np.random.default_rng(16384)
    heads = sorted({0, 1, H // 2 - 1, H - 1, *rng.integers(0, H, 4).tolist()})
    sel = torch.as_tensor(heads, device=dev)
    cpu = [t.index_select(1, sel).double().cpu().numpy() for t in (q, k, v, do)]
    ref = oracle.packed_forward(d, *cpu[:3], scale)
    np.testing.assert_allclose(to64(out.index_select(1, sel)), ref["final_out"], rtol=0, atol=O_TOL)
    np.testing.assert_allclose(to64(lse.index_select(1, sel)), ref["final_lse"], rtol=0, atol=LSE_TOL)
    for b in range(2):
        np.testing.assert_allclose(to64(o_part_shard[b].index_select(1, sel)), ref["o_part"][b, 1170:],
                                   rtol=0, atol=O_TOL)
        np.testing.assert_allclose(to64(lse_part_shard[b].index_select(1, sel)), ref["lse_part"][b, 1170:],
                                   rtol=0, atol=LSE_TOL)
    rq, rk, rv = oracle.packed_backward(d, *cpu[:3], cpu[3], scale)
    _check_bwd(dq.index_select(1, sel), rq, "dq")
    _check_bwd(dk.index_select(1, sel), rk, "dk")
    _check_bwd(dv.index_select(1, sel), rv, "dv")
