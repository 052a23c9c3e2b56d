"""Ring steps at full size: the coalesced whole+shard batch (a 9450-query
shard against 8 K/V blocks of 9450 tokens, six whole 1560-token fillers, 40
heads, d=128) run as eight forward steps (zl_attn_fwd_step, fillers spread
over the steps) and eight backward steps (zl_attn_bwd_step, fillers in the
last step), exactly as bench.py --mode ring launches them, checked against
the all-blocks launch of the same inputs (which the full-size oracle tests
check against the oracle):

  * forward: the shard rows after the last step and every filler row match
    the all-blocks output plus LSE merge to the forward tolerances (the ring
    folds blocks one by one into a running fp32 (O, LSE), the all-blocks
    path merges fp32 partials: the same sum in a different order);
  * backward: every block's dK/dV and the fillers' dQ/dK/dV are the same work
    items on the same inputs and match bit for bit; the shard's dQ, summed
    block by block in fp32, matches to the backward tolerances.
"""
import numpy as np
import pytest
import torch

import bench
from paper_2608_01150_amd import workloads as W
from tests._gpu import HAVE_GPU, api, to64

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="needs a GPU")]

O_TOL, LSE_TOL = 2e-2, 1e-3


def test_coalesced_batch_ring_steps_match_all_blocks():
    w = W.get("c4")
    dev = torch.device("cuda:0")
    H, hd = w.num_heads, w.head_dim
    desc = api.SegDesc.of(w)
    q, k, v, do = (w.full(t, device=dev) for t in (W.TENSOR_Q, W.TENSOR_K, W.TENSOR_V, W.TENSOR_DO))
    out, lse, o_part, lse_part = api.attn_fwd(desc, q, k, v, w.scale)
    api.lse_merge(desc, o_part, lse_part, out, lse)
    dq_ref, dk_ref, dv_ref = api.attn_bwd(desc, q, k, v, out, lse, do, w.scale)
    torch.cuda.synchronize()
    del o_part, lse_part

    # forward ring steps
    steps = bench.ring_steps(w, q, k, v)
    R = len(steps)
    n_sq = steps[0]["n_shard_rows"]
    max_tq = max(st["q"].shape[0] for st in steps)
    o_acc = torch.empty((max_tq, H, hd), dtype=torch.float32, device=dev)
    lse_acc = torch.empty((max_tq, H), dtype=torch.float32, device=dev)
    for r, st in enumerate(steps):
        flags = (api.ZL_STEP_FIRST if r == 0 else 0) | (api.ZL_STEP_LAST if r == R - 1 else 0)
        api.attn_fwd_step(st["desc"], st["q"], st["k"], st["v"], w.scale, st["out"], st["lse"], o_acc, lse_acc, flags)
    torch.cuda.synchronize()
    last = steps[-1]
    assert (last["out"][:n_sq].float() - out[:n_sq].float()).abs().max().item() <= O_TOL
    assert (last["lse"][:n_sq] - lse[:n_sq]).abs().max().item() <= LSE_TOL
    # fillers: step r carries WHOLE filler i (segment 1 + i) when i % R == r, right after the shard rows
    wholes = list(range(1, w.num_segments))
    for r, st in enumerate(steps):
        row = n_sq
        for i, s in enumerate(wholes):
            if i % R != r:
                continue
            a, b = w.cu_seqlens_q[s], w.cu_seqlens_q[s + 1]
            n = b - a
            assert (st["out"][row:row + n].float() - out[a:b].float()).abs().max().item() <= O_TOL
            assert (st["lse"][row:row + n] - lse[a:b]).abs().max().item() <= LSE_TOL
            row += n
    del steps, o_acc, lse_acc

    # backward ring steps, in place on the full tensors
    dq = torch.full_like(q, float("nan"))
    dk = torch.full_like(k, float("nan"))
    dv = torch.full_like(v, float("nan"))
    dq_acc = torch.empty((n_sq, H, hd), dtype=torch.float32, device=dev)
    ws = torch.empty(api.workspace_size(desc, H, hd, q.dtype, api.ZL_OP_BWD), dtype=torch.uint8, device=dev)
    for b in bench.ring_bwd_steps(w, q, k, v, out, lse, do, dq, dk, dv):
        api.attn_bwd_step(b["desc"], b["q"], b["k"], b["v"], b["out"], b["lse"], b["do"], w.scale, b["dq"], b["dk"],
                          b["dv"], dq_acc, b["flags"], ws)
    torch.cuda.synchronize()
    assert torch.equal(dk, dk_ref) and torch.equal(dv, dv_ref)
    assert torch.equal(dq[n_sq:], dq_ref[n_sq:])
    got, ref = to64(dq[:n_sq]), to64(dq_ref[:n_sq])
    assert np.abs(got - ref).max() <= 2e-2 * max(1.0, np.abs(ref).max())
    assert np.linalg.norm(got - ref) / np.linalg.norm(ref) <= 2e-2
