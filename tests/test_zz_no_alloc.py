"""zl_attn_bwd_noalloc, the backward for callers that cannot allocate: its work tables and workspace
sit in the library's static device scratch.  It must give zl_attn_bwd's results bit for bit (the same
work items on the same kernels) on consecutive calls that reuse the scratch, the second one smaller
and the third with more work items than resident workgroups, and reject a batch that does not fit the
scratch before enqueueing anything."""
import numpy as np
import pytest
import torch

from tests import _descs
from tests._gpu import HAVE_GPU, api

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="needs a GPU")]


def _inputs(d, H, hd, seed):
    g = torch.Generator().manual_seed(seed)
    tq, tk = d["cu_seqlens_q"][-1], d["cu_seqlens_k"][-1]
    return [torch.randn((n, H, hd), generator=g).to(torch.bfloat16).cuda() for n in (tq, tk, tk, tq)]


def _compare(d, H, hd, seed):
    desc = api.SegDesc.of(d)
    q, k, v, do = _inputs(d, H, hd, seed)
    scale = hd ** -0.5
    out, lse, o_part, lse_part = api.attn_fwd(desc, q, k, v, scale)
    if desc.num_slots:
        api.lse_merge(desc, o_part, lse_part, out, lse)
    nan = float("nan")
    ref = [torch.full_like(t, nan) for t in (q, k, v)]
    api.attn_bwd(desc, q, k, v, out, lse, do, scale, *ref)
    got = [torch.full_like(t, nan) for t in (q, k, v)]
    api.attn_bwd_noalloc(desc, q, k, v, out, lse, do, scale, *got)
    torch.cuda.synchronize()
    for name, a, b in zip(("dq", "dk", "dv"), got, ref):
        assert not torch.isnan(b).any(), name
        assert torch.equal(a, b), f"{name} differs from zl_attn_bwd"


def test_noalloc_backward_matches_backward_on_consecutive_calls():
    # first call: whole, empty whole, whole, a three-block shard (one block empty), a one-block shard
    _compare(_descs.mixed_small(), 3, 128, 71)
    # second call, smaller: the scratch still holds the first call's tables and workspace
    small = _descs.desc(cu_q=(0, 90, 130), kind=(0, 1), kv_first=(0, 1), kv_count=(1, 2),
                        cu_k=(0, 90, 140, 170), block_index=(0, 1, 0), num_slots=2)
    _compare(small, 2, 64, 72)
    # third call, 96 heads: 864 dK/dV and 384 dQ items, more than the GPU's resident workgroups, so most
    # items are handed out at run time through the kernels' work queues
    _compare(_descs.mixed_small(), 96, 128, 73)


def test_noalloc_rejects_a_batch_beyond_the_scratch():
    """8 bytes of workspace per (row, head): 66,000 rows x 64 heads need 33.8 MB > 32 MiB.  The call
    fails before enqueueing anything (the tensors are never read)."""
    H, hd, n = 64, 64, 66000
    d = _descs.desc(cu_q=(0, n), kind=(0,), kv_first=(0,), kv_count=(1,), cu_k=(0, n), block_index=(0,),
                    num_slots=0)
    desc = api.SegDesc.of(d)
    t = [torch.empty((n, H, hd), dtype=torch.bfloat16, device="cuda") for _ in range(8)]
    lse = torch.empty((n, H), dtype=torch.float32, device="cuda")
    with pytest.raises(api.ZlError) as e:
        api.attn_bwd_noalloc(desc, t[0], t[1], t[2], t[3], lse, t[4], hd ** -0.5, t[5], t[6], t[7])
    assert e.value.status == api.ZL_ERR_WORKSPACE and "static scratch" in str(e.value)
    torch.cuda.synchronize()
