"""HIP graph capture of the attention path.  Once a descriptor's schedule is
cached (an eager first call), the library's calls only launch kernels, so a
forward + merge + backward sequence can be captured and replayed.  The graph
is replayed several times, with the outputs refilled with NaN and unrelated
eager work (another forward, a synchronize) between replays, and every replay
must equal the eager result bit for bit (the kernels are deterministic)."""
import pytest
import torch

from tests import _descs
from tests._gpu import HAVE_GPU, api

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="needs a GPU")]


def test_captured_forward_merge_backward_replays_match_eager():
    dev = torch.device("cuda:0")
    d = _descs.mixed_small()
    desc = api.SegDesc.of(d)
    H, hd, scale = 3, 128, 128 ** -0.5
    g = torch.Generator().manual_seed(20261202)
    tq, tk = d["cu_seqlens_q"][-1], d["cu_seqlens_k"][-1]
    q, k, v, do = (torch.randn((n, H, hd), generator=g).to(torch.bfloat16).to(dev) for n in (tq, tk, tk, tq))
    api.profile_enable(False)

    # eager reference (also caches the forward, merge and backward schedules)
    out, lse, o_part, lse_part = api.attn_fwd(desc, q, k, v, scale)
    api.lse_merge(desc, o_part, lse_part, out, lse)
    dq, dk, dv = api.attn_bwd(desc, q, k, v, out, lse, do, scale)
    torch.cuda.synchronize()

    # static buffers of the graph
    out_g, lse_g = torch.empty_like(out), torch.empty_like(lse)
    op_g, lp_g = torch.empty_like(o_part), torch.empty_like(lse_part)
    dq_g, dk_g, dv_g = torch.empty_like(dq), torch.empty_like(dk), torch.empty_like(dv)
    ws = torch.empty(api.workspace_size(desc, H, hd, torch.bfloat16, api.ZL_OP_BWD), dtype=torch.uint8, device=dev)

    def body():
        api.attn_fwd(desc, q, k, v, scale, out_g, lse_g, op_g, lp_g)
        api.lse_merge(desc, op_g, lp_g, out_g, lse_g)
        api.attn_bwd(desc, q, k, v, out_g, lse_g, do, scale, dq_g, dk_g, dv_g, ws)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        body()  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        body()

    bufs = (out_g, lse_g, dq_g, dk_g, dv_g)
    refs = (out, lse, dq, dk, dv)
    other = torch.empty_like(out)
    # More descriptors than the work-table cache once held (64), each with its own tables: no call may
    # free a table the graph captured (the cache keeps every table until zl_shutdown).
    for n in range(1, 81):
        dn = api.SegDesc([0, n], [0], [0], [1], [0, n], [0], 0)
        xn = torch.randn((n, 1, 64), dtype=torch.bfloat16, device=dev)
        api.attn_fwd(dn, xn, xn, xn, 0.125)
    torch.cuda.synchronize()
    for rep in range(3):
        for b in bufs:
            b.fill_(float("nan"))
        api.attn_fwd(desc, do, k, v, scale, other)  # unrelated eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for name, got, ref in zip(("out", "lse", "dq", "dk", "dv"), bufs, refs):
            assert torch.equal(got, ref), f"replay {rep}: {name} differs from the eager result"
