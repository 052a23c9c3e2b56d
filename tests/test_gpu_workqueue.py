"""Dynamic work distribution of the persistent kernels (forward, dK/dV, dQ).

A launch with more work items than the GPU has resident workgroups hands out
its items through per-XCD queues with device-scope atomic counters (the
first round by workgroup index, the rest claimed at run time, faster XCDs
taking over the tail of slower ones).  Which workgroup runs an item must not
change any value: every item's computation is independent of the others and
each output element is written by exactly one item.  So

* the outputs equal, bit for bit, those of the same batch run with one item
  per workgroup in dispatch order (ZL_STATIC_DISPATCH=1, in a child process,
  since the switch is read once per process);
* back-to-back launches into NaN-filled outputs give the same bits every time
  (each launch's last workgroup must leave the counters at zero, or the next
  launch would skip items and leave NaN behind);
* launches of the same batch on several streams at once give the same bits
  (each stream has its own counters).
"""
import os
import subprocess
import sys
import tempfile

import numpy as np
import pytest
import torch

from paper_2608_01150_amd import workloads as W
from tests._gpu import HAVE_GPU, api

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="needs a GPU")]

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def batch(head_dim=128):
    """WHOLE segments of ragged lengths plus a three-block SHARD, 48 heads:
    768 forward, 1104 dK/dV and 576 dQ items, all above the 256 CUs."""
    segs = [("whole", 600, 0), ("whole", 1000, 10_000), ("whole", 333, 20_000), ("whole", 64, 30_000),
            ("shard", 300, 40_000, [(200, 40_000, 0), (250, 50_000, 1), (130, 60_000, 2)])]
    return W.build_segments("workqueue-test", 48, head_dim, segs, 20261202)


def inputs(w, dev):
    return tuple(w.full(t, device=dev) for t in (W.TENSOR_Q, W.TENSOR_K, W.TENSOR_V, W.TENSOR_DO))


def alloc(w, desc, dev):
    """NaN-filled outputs (rows a launch does not write stay NaN in every run) and the workspace."""
    tq, tk, H, hd = w.total_q, w.total_k, w.num_heads, w.head_dim
    nan = float("nan")
    b = dict(out=torch.full((tq, H, hd), nan, dtype=torch.bfloat16, device=dev),
             lse=torch.full((tq, H), nan, dtype=torch.float32, device=dev),
             o_part=torch.full((w.num_slots, tq, H, hd), nan, dtype=torch.float32, device=dev),
             lse_part=torch.full((w.num_slots, tq, H), nan, dtype=torch.float32, device=dev),
             dq=torch.full((tq, H, hd), nan, dtype=torch.bfloat16, device=dev),
             dk=torch.full((tk, H, hd), nan, dtype=torch.bfloat16, device=dev),
             dv=torch.full((tk, H, hd), nan, dtype=torch.bfloat16, device=dev))
    ws = torch.empty(api.workspace_size(desc, H, hd, torch.bfloat16, api.ZL_OP_BWD), dtype=torch.uint8, device=dev)
    return b, ws


def refill(b):
    for t in b.values():
        t.fill_(float("nan"))


def run(w, desc, q, k, v, do, b, ws):
    """Forward, merge and backward into the buffers b."""
    api.attn_fwd(desc, q, k, v, w.scale, b["out"], b["lse"], b["o_part"], b["lse_part"])
    api.lse_merge(desc, b["o_part"], b["lse_part"], b["out"], b["lse"])
    api.attn_bwd(desc, q, k, v, b["out"], b["lse"], do, w.scale, b["dq"], b["dk"], b["dv"], ws)
    return b


def bits(t):
    t = t.detach().contiguous().cpu()
    return t.view(torch.int16).numpy() if t.dtype == torch.bfloat16 else t.view(torch.int32).numpy()


def check_equal(ref, got, what):
    for n, t in ref.items():
        a, b = bits(t), bits(got[n])
        assert np.array_equal(a, b), f"{what}: {n} differs in {(a != b).sum()} of {a.size} elements"


@pytest.mark.parametrize("head_dim", [128, 64])
def test_dynamic_dispatch_equals_static_dispatch(head_dim):
    dev = torch.device("cuda:0")
    w = batch(head_dim)
    desc = api.SegDesc.of(w)
    items, _ = api.plan_dump(desc, w.num_heads, w.head_dim, torch.bfloat16, api.ZL_OP_FWD)
    assert len(items) > torch.cuda.get_device_properties(0).multi_processor_count, "batch must exceed one round"
    ref = run(w, desc, *inputs(w, dev), *alloc(w, desc, dev))
    torch.cuda.synchronize()
    with tempfile.TemporaryDirectory() as tmp:
        path = os.path.join(tmp, "static.npz")
        env = dict(os.environ, ZL_STATIC_DISPATCH="1")
        r = subprocess.run([sys.executable, "-m", "tests.test_gpu_workqueue", path, str(head_dim)], cwd=ROOT, env=env,
                           capture_output=True, text=True, timeout=600)
        assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
        st = np.load(path)
        for n, t in ref.items():
            a, b = bits(t), st[n]
            assert np.array_equal(a, b), f"{n}: dynamic and static dispatch differ in {(a != b).sum()} elements"


def test_back_to_back_launches_leave_counters_at_zero():
    dev = torch.device("cuda:0")
    w = batch()
    desc = api.SegDesc.of(w)
    q, k, v, do = inputs(w, dev)
    ref = run(w, desc, q, k, v, do, *alloc(w, desc, dev))
    b, ws = alloc(w, desc, dev)
    for i in range(12):
        refill(b)
        run(w, desc, q, k, v, do, b, ws)
        torch.cuda.synchronize()
        check_equal(ref, b, f"launch {i}")


def test_concurrent_streams_have_their_own_counters():
    dev = torch.device("cuda:0")
    w = batch()
    desc = api.SegDesc.of(w)
    q, k, v, do = inputs(w, dev)
    ref = run(w, desc, q, k, v, do, *alloc(w, desc, dev))
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in range(4)]
    bufs = [alloc(w, desc, dev) for _ in streams]
    for rep in range(3):
        for b, _ in bufs:
            refill(b)
        torch.cuda.synchronize()
        for st, (b, ws) in zip(streams, bufs):
            with torch.cuda.stream(st):
                run(w, desc, q, k, v, do, b, ws)
        torch.cuda.synchronize()
        for j, (b, _) in enumerate(bufs):
            check_equal(ref, b, f"round {rep}, stream {j}")


if __name__ == "__main__":
    # Child process of test_dynamic_dispatch_equals_static_dispatch (run with ZL_STATIC_DISPATCH=1).
    dev = torch.device("cuda:0")
    w = batch(int(sys.argv[2]))
    desc = api.SegDesc.of(w)
    res = run(w, desc, *inputs(w, dev), *alloc(w, desc, dev))
    torch.cuda.synchronize()
    np.savez(sys.argv[1], **{n: bits(t) for n, t in res.items()})
