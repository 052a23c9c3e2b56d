"""Benchmark of the packed whole+shard attention hot path on one MI355X.

One step = the whole path over one packed batch: one forward launch over the
WHOLE and SHARD segments together, the LSE merge of the shard partials (when
the batch has shards), and the backward (preprocess, dK/dV, dQ), inputs
resident in HBM.  The default workload is the mixed image-video batch: one
32,760-token 480p video, two 3600-token and eight 1560-token images, all
whole, coalesced into one block-diagonal launch (Sec. IV-D), 40 heads, d=128,
bf16, the video's Q and K scaled by 4.  It has no shards, so the same run also
times the LSE merge on the coalesced whole+shard batch (one GPU's share of a
75,600-token video at CP=8: a 9450-query shard's 8 block partials), reported
as merge_kernel with its own workload name.

Prints one JSON line.  value = fwd+bwd TFLOP/s with the FlashAttention FLOP
convention (forward 4*d*H*pairs, backward 10*d*H*pairs, pairs = block-diagonal
query-key pairs only).  roofline = the dominant (longest) kernel, timed with
HIP events on the stream it is launched on inside the timed region, priced at
its share of the algorithmic FLOPs (no recompute: forward S and PV 4*d per
pair, dK/dV kernel dP, dV, dK 6*d, dQ kernel dQ 2*d; 12*d per step) against
the bf16 dense MFMA peak; the executed rate (4, 8, 6 *d, recompute included)
and its fraction of a bf16 GEMM measured in the same run stand beside it.
cpu_baseline = the fp64 oracle timed on this host's cores on a bounded
sample of the same batch (see --cpu-seconds).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

METRIC = "packed whole+shard attention fwd+bwd TFLOP/s (bf16) and % of MFMA peak"
BF16_PEAK_TFLOPS = 2516.6      # 256 CU x 2.4 GHz x 4096 bf16 FLOP/clk/CU (dense)
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c3", help="c2..c5 (default c3: mixed image-video batch)")
    ap.add_argument("--merge-workload", default="c4",
                    help="when the workload has no shards: the batch whose LSE merge is timed in the same run")
    ap.add_argument("--merge-reps", type=int, default=20, help="timed merge launches on --merge-workload")
    ap.add_argument("--no-ceiling", action="store_true", help="skip the bf16 GEMM ceiling measurement")
    ap.add_argument("--ulysses-group", type=int, default=8, help="group size h for --mode ulysses")
    ap.add_argument("--partials", default="fp32", choices=("fp32", "bf16"),
                    help="--mode blocks: dtype of the shard partials between the forward and the merge "
                         "(bf16 halves their bytes and rounds each block's output once more)")
    ap.add_argument("--mode", default="blocks", choices=("blocks", "ring", "gather", "ulysses"),
                    help="how a shard's K/V blocks reach the forward: blocks = all blocks in one launch plus "
                         "the LSE merge (default); ring = one ring step per block with the merge fused into "
                         "the epilogue (fillers spread over the steps) and one backward step per block with "
                         "dQ accumulated across the steps (fillers in the last); gather = one launch against the "
                         "concatenated blocks (all-gather), no partials and no merge; ulysses = one GPU's "
                         "share of the batch's WHOLE sequences under Ulysses (1,h,1): QKV pack, unpack, "
                         "attention on H/h heads over the full sequences, output pack and unpack (the two "
                         "all-to-alls are RCCL's and not run here: the send buffer stands in for the receive)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="accumulate oracle heads until this much CPU time is spent")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB (for scaling HBM byte counters)")
    return ap.parse_args()


# CPU baseline sample: a shard keeps the first 1/SHARD_DIV of its query rows, a whole segment longer
# than LONG_WHOLE the first 1/LONG_DIV (each against all of its keys).
LONG_WHOLE, SHARD_DIV, LONG_DIV = 8192, 9, 27


def cpu_baseline(w, min_seconds):
    """Time the oracle (as it stands) on a bounded sample of workload w.

    Sample: heads taken one at a time until at least `min_seconds` of oracle
    time has accumulated (or every head is done); per head, every whole
    segment of up to LONG_WHOLE tokens in full (forward + backward), each
    shard reduced to its first 1/SHARD_DIV of query rows and each longer
    whole segment to its first 1/LONG_DIV, forward against all of its keys
    (blocks), merge, backward.  FLOPs are counted with the same convention as
    the GPU value (14*d per pair).
    """
    import numpy as np
    import oracle
    from paper_2608_01150_amd import workloads as W

    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [os.cpu_count() or 1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count() or 1
    d = w.desc_dict()
    cq = list(d["cu_seqlens_q"])
    new_cq, rows, kinds = [0], [], list(d["kind"])
    for s in range(w.num_segments):
        a, b = cq[s], cq[s + 1]
        if w.kind[s] == W.SHARD or b - a > LONG_WHOLE:
            div = SHARD_DIV if w.kind[s] == W.SHARD else LONG_DIV
            b = a + (b - a + div - 1) // div
            kinds[s] = W.SHARD   # a query subset against all of the segment's keys
        rows.append((a, b))
        new_cq.append(new_cq[-1] + (b - a))
    d2 = dict(d, cu_seqlens_q=tuple(new_cq), kind=tuple(kinds), num_slots=max(1, d["num_slots"]))
    pairs = 0
    for s in range(w.num_segments):
        lq = new_cq[s + 1] - new_cq[s]
        for j in range(w.kv_first[s], w.kv_first[s] + w.kv_count[s]):
            pairs += lq * (w.cu_seqlens_k[j + 1] - w.cu_seqlens_k[j])
    spent, heads = 0.0, 0
    while heads < w.num_heads and spent < min_seconds:
        hs = [heads]
        q = np.concatenate([w.slice(W.TENSOR_Q, a, b, heads=hs).double().numpy() for a, b in rows])
        do = np.concatenate([w.slice(W.TENSOR_DO, a, b, heads=hs).double().numpy() for a, b in rows])
        k = w.slice(W.TENSOR_K, 0, w.total_k, heads=hs).double().numpy()
        v = w.slice(W.TENSOR_V, 0, w.total_k, heads=hs).double().numpy()
        t0 = time.perf_counter()
        fwd = oracle.packed_forward(d2, q, k, v, w.scale)
        for s in range(w.num_segments):
            if w.kind[s] == W.SHARD:
                a, b = new_cq[s], new_cq[s + 1]
                oracle.lse_merge(fwd["o_part"][:, a:b, 0], fwd["lse_part"][:, a:b, 0])
        oracle.packed_backward(d2, q, k, v, do, w.scale)
        spent += time.perf_counter() - t0
        heads += 1
    flops = 14.0 * w.head_dim * heads * pairs
    return {"value": flops / spent / 1e12, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{heads} of {w.num_heads} heads; whole segments up to {LONG_WHOLE} tokens in full, the first "
                      f"1/{SHARD_DIV} of each shard's query rows and the first 1/{LONG_DIV} of each longer whole "
                      f"segment's, against all of their keys; fwd+merge+bwd fp64; {pairs} pairs/head, {spent:.1f} s"}


def gathered_descriptor(w):
    """The batch with each SHARD segment's consecutive K/V ranges merged into one range (the K/V an
    all-gather delivers): no partial slots, no merge."""
    import numpy as np
    cu_k = [0]
    kv_first, kv_count, bidx = [], [], []
    for s in range(w.num_segments):
        j0, j1 = w.kv_first[s], w.kv_first[s] + w.kv_count[s]
        kv_first.append(len(cu_k) - 1)
        kv_count.append(1)
        cu_k.append(cu_k[-1] + int(w.cu_seqlens_k[j1] - w.cu_seqlens_k[j0]))
        bidx.append(0)
    return dict(cu_seqlens_q=np.asarray(w.cu_seqlens_q, np.int32), kind=np.asarray(w.kind, np.uint8),
                kv_first=np.asarray(kv_first, np.int32), kv_count=np.asarray(kv_count, np.int32),
                cu_seqlens_k=np.asarray(cu_k, np.int32), block_index=np.asarray(bidx, np.int32), num_slots=1,
                q_offset=None, k_offset=None)


def ring_steps(w, q, k, v):
    """Per-step packed inputs of the ring: step r carries block r of every shard (shard rows first, so
    the accumulator rows line up) and the WHOLE fillers with index % R == r."""
    import numpy as np
    import torch
    from paper_2608_01150_amd import api
    from paper_2608_01150_amd import workloads as W
    shards = [s for s in range(w.num_segments) if w.kind[s] == W.SHARD]
    wholes = [s for s in range(w.num_segments) if w.kind[s] == W.WHOLE]
    R = w.kv_count[shards[0]]
    assert all(w.kv_count[s] == R for s in shards), "ring mode needs every shard to have the same block count"
    rows = lambda s: (int(w.cu_seqlens_q[s]), int(w.cu_seqlens_q[s + 1]))
    krows = lambda j: (int(w.cu_seqlens_k[j]), int(w.cu_seqlens_k[j + 1]))
    n_sq = sum(b - a for a, b in map(rows, shards))
    out = []
    for r in range(R):
        segs = shards + [s for i, s in enumerate(wholes) if i % R == r]
        lq = [rows(s)[1] - rows(s)[0] for s in segs]
        ranges = [krows(w.kv_first[s] + (r if w.kind[s] == W.SHARD else 0)) for s in segs]
        lk = [b - a for a, b in ranges]
        n = len(segs)
        desc = api.SegDesc(np.concatenate([[0], np.cumsum(lq)]).astype(np.int32),
                           np.asarray([w.kind[s] for s in segs], np.uint8), np.arange(n, dtype=np.int32),
                           np.ones(n, np.int32), np.concatenate([[0], np.cumsum(lk)]).astype(np.int32),
                           np.zeros(n, np.int32), 1)
        qr = torch.cat([q[slice(*rows(s))] for s in segs])
        kr = torch.cat([k[a:b] for a, b in ranges])
        vr = torch.cat([v[a:b] for a, b in ranges])
        out.append(dict(desc=desc, q=qr, k=kr, v=vr, out=torch.empty_like(qr),
                        lse=torch.empty((qr.shape[0], q.shape[1]), dtype=torch.float32, device=q.device),
                        n_shard_rows=n_sq))
    return out


def ring_bwd_steps(w, q, k, v, out, lse, do, dq, dk, dv):
    """Backward ring steps over the packed batch: step r brings block r of the (single, leading) shard,
    and the last step also carries every WHOLE filler, whose K/V rows follow the last block.  Every step
    works on views of the full tensors (the shard's rows are the first rows), so dK/dV and dQ land in
    place."""
    import numpy as np
    from paper_2608_01150_amd import api
    from paper_2608_01150_amd import workloads as W
    assert w.kind[0] == W.SHARD and all(kd == W.WHOLE for kd in w.kind[1:]), "ring backward: one leading shard"
    R = w.kv_count[0]
    n_sq = int(w.cu_seqlens_q[1])
    cu_k = [int(x) for x in w.cu_seqlens_k]
    steps = []
    for r in range(R):
        last = r == R - 1
        nseg = w.num_segments if last else 1
        rows = w.total_q if last else n_sq
        b0 = cu_k[w.kv_first[0] + r]
        k_end = w.total_k if last else cu_k[w.kv_first[0] + r + 1]
        lk = [cu_k[w.kv_first[0] + r + 1] - b0] + [cu_k[w.kv_first[s] + 1] - cu_k[w.kv_first[s]]
                                                    for s in range(1, nseg)]
        desc = api.SegDesc(np.asarray(w.cu_seqlens_q[:nseg + 1], np.int32),
                           np.asarray(w.kind[:nseg], np.uint8), np.arange(nseg, dtype=np.int32),
                           np.ones(nseg, np.int32), np.concatenate([[0], np.cumsum(lk)]).astype(np.int32),
                           np.zeros(nseg, np.int32), 1)
        sl, ks = slice(0, rows), slice(b0, k_end)
        steps.append(dict(desc=desc, q=q[sl], out=out[sl], lse=lse[sl], do=do[sl], dq=dq[sl], k=k[ks], v=v[ks],
                          dk=dk[ks], dv=dv[ks],
                          flags=(api.ZL_STEP_FIRST if r == 0 else 0) | (api.ZL_STEP_LAST if last else 0)))
    return steps


# Source files whose text (with the compile flags applied to them) determines
# each kernel's code; a stored counter measurement applies only while their
# hash is unchanged.
KERNEL_SOURCES = {
    "fwd": ["fwd_bf16.hip"],
    "bwd_dkdv": ["bwd_bf16.hip"],
    "bwd_dq": ["bwd_bf16.hip"],
    "merge": ["merge.hip"],
}
COMMON_SOURCES = ["zl_device.h", "zl_internal.h"]
TRAFFIC_FILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "traffic.json")


def kernel_source_hash(kernel: str) -> str:
    import hashlib
    csrc = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2608_01150_amd", "csrc")
    from paper_2608_01150_amd import build as _build
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel] + COMMON_SOURCES:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    flags = [a for a in _build.HIP_FLAGS if not a.startswith("/")]  # include paths vary by checkout
    for f in KERNEL_SOURCES[kernel]:
        flags += getattr(_build, "FILE_FLAGS", {}).get(f, [])
    h.update("\0".join(flags).encode())
    return h.hexdigest()


def stored_traffic(kernel: str, workload: str):
    """HBM bytes per launch measured with rocprofv3 FETCH_SIZE / WRITE_SIZE (copy-calibrated)
    for this kernel and workload ({kernel: {workload name: record}} in the file), or None if absent
    or taken on different kernel source."""
    try:
        with open(TRAFFIC_FILE) as fh:
            rec = json.load(fh).get(kernel, {}).get(workload)
    except (OSError, ValueError, AttributeError):
        return None
    if not rec or rec.get("src_sha256") != kernel_source_hash(kernel):
        return None
    return rec


def merge_on(name, reps, partials):
    """Times the LSE merge on workload `name` (one forward fills its partials, then `reps` merge
    launches); returns the merge_kernel record.  Used when the benchmarked batch has no shards."""
    import torch
    from paper_2608_01150_amd import api
    from paper_2608_01150_amd import workloads as W
    w = W.get(name)
    dev = torch.device("cuda:0")
    desc = api.SegDesc.of(w)
    H, hd = w.num_heads, w.head_dim
    q, k, v = (w.full(t, device=dev) for t in (W.TENSOR_Q, W.TENSOR_K, W.TENSOR_V))
    pdt = torch.bfloat16 if partials == "bf16" else torch.float32
    out = torch.empty_like(q)
    lse = torch.empty((w.total_q, H), dtype=torch.float32, device=dev)
    o_part = torch.empty((w.num_slots, w.total_q, H, hd), dtype=pdt, device=dev)
    lse_part = torch.empty((w.num_slots, w.total_q, H), dtype=torch.float32, device=dev)
    api.attn_fwd(desc, q, k, v, w.scale, out, lse, o_part, lse_part)
    for _ in range(3):
        api.lse_merge(desc, o_part, lse_part, out, lse)
    torch.cuda.synchronize()
    api.profile_reset()
    api.profile_enable(True)
    for _ in range(reps):
        api.lse_merge(desc, o_part, lse_part, out, lse)
    torch.cuda.synchronize()
    api.profile_enable(False)
    ms_total, n = api.profile_read(api.ZL_K_MERGE)
    rec = merge_record(w, H, hd, partials, ms_total / n)
    rec.update(workload=w.name, launches=n)
    del q, k, v, out, lse, o_part, lse_part
    torch.cuda.empty_cache()
    return rec


def merge_record(w, H, hd, partials, ms):
    from paper_2608_01150_amd import workloads as W
    sr = w.shard_rows()
    nb = max(w.kv_count[s] for s in range(w.num_segments) if w.kind[s] == W.SHARD)
    pb = 2 if partials == "bf16" else 4   # bytes per partial element
    mbytes = H * sr * (nb * (pb * hd + 4) + 2 * hd + 4)
    gbs = mbytes / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(gbs / HBM_PEAK_GBS, 4), "bytes": mbytes, "ms": round(ms, 4)}


def hbm_ceilings(mib=1024, reps=10):
    """HBM rates measured on this GPU in this run, as ceilings for HBM-bound kernels such as the merge
    (which reads 96% of its bytes): a device copy (torch copy_, read + write bytes) and a read-only
    reduction (torch sum), each over `mib` MiB of fp32."""
    import torch
    src = torch.ones((mib << 20) // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    nbytes = mib << 20

    def rate(fn, moved):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(reps):
            fn()
        t1.record()
        torch.cuda.synchronize()
        return round(moved / (t0.elapsed_time(t1) / reps * 1e-3) / 1e9, 1)

    out = {"copy_gbs": rate(lambda: dst.copy_(src), 2 * nbytes), "read_gbs": rate(lambda: src.sum(), nbytes),
           "kind": f"{mib} MiB fp32: torch copy_ (read + write) and torch sum (read)"}
    del src, dst
    return out


def gemm_ceiling(n=8192, reps=10):
    """bf16 GEMM rate (torch.matmul, hipBLASLt) on this GPU in this run: a measured ceiling for dense
    bf16 MFMA work with no attention dependencies."""
    import torch
    a = torch.randn((n, n), device="cuda:0").to(torch.bfloat16)
    b = torch.randn((n, n), device="cuda:0").to(torch.bfloat16)
    for _ in range(3):
        c = a @ b
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(reps):
        c = a @ b
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / reps
    del a, b, c
    return {"kind": f"bf16 GEMM {n}^3 (torch.matmul, hipBLASLt)", "tflops": round(2.0 * n ** 3 / (ms * 1e-3) / 1e12, 1)}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: it measures one GPU's share of the batch "
              "(context parallelism is simulated by feeding that GPU's K/V blocks locally); "
              "--gpus must be 1.", file=sys.stderr)
        sys.exit(2)
    import torch
    if args.copy_calibration_mib:
        n = args.copy_calibration_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n}), flush=True)
        return
    from paper_2608_01150_amd import api
    from paper_2608_01150_amd import workloads as W

    w = W.get(args.workload)
    if args.mode in ("ring", "gather") and not any(w.kind[s] == W.SHARD for s in range(w.num_segments)):
        print(f"--mode {args.mode} delivers a shard's K/V blocks step by step or concatenated; the workload "
              f"{w.name} has no shard segments (use --workload c4 or c5).", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    desc = api.SegDesc.of(w)
    H, hd = w.num_heads, w.head_dim
    q = w.full(W.TENSOR_Q, device=dev)
    k = w.full(W.TENSOR_K, device=dev)
    v = w.full(W.TENSOR_V, device=dev)
    do = w.full(W.TENSOR_DO, device=dev)
    out = torch.empty_like(q)
    lse = torch.empty((w.total_q, H), dtype=torch.float32, device=dev)
    o_part = lse_part = None
    if w.num_slots:
        pdt = torch.bfloat16 if args.partials == "bf16" else torch.float32
        o_part = torch.empty((w.num_slots, w.total_q, H, hd), dtype=pdt, device=dev)
        lse_part = torch.empty((w.num_slots, w.total_q, H), dtype=torch.float32, device=dev)
    dq = torch.empty_like(q)
    dk = torch.empty_like(k)
    dv = torch.empty_like(v)
    ws = torch.empty(api.workspace_size(desc, H, hd, q.dtype, api.ZL_OP_BWD), dtype=torch.uint8, device=dev)

    def step():
        api.attn_fwd(desc, q, k, v, w.scale, out, lse, o_part, lse_part)
        if w.num_slots:
            api.lse_merge(desc, o_part, lse_part, out, lse)
        api.attn_bwd(desc, q, k, v, out, lse, do, w.scale, dq, dk, dv, ws)

    if args.mode == "ulysses":
        G = args.ulysses_group
        assert all(kd == W.WHOLE for kd in w.kind) and H % G == 0, "ulysses mode: a WHOLE-only batch, H % h == 0"
        Hl = H // G
        lens = [int(w.cu_seqlens_q[s + 1] - w.cu_seqlens_q[s]) for s in range(w.num_segments)]
        # even shards (the first ones one longer where a length does not divide)
        shard = [[n // G + (1 if j < n % G else 0) for n in lens] for j in range(G)]
        import numpy as np
        cu_rank = np.array([np.concatenate([[0], np.cumsum(sh)]) for sh in shard], np.int32)
        t_local = int(cu_rank[0][-1])
        t_full = w.total_q
        ql, kl, vl = q[:t_local], k[:t_local], v[:t_local]      # this rank's local rows (any rows of the right shape)
        send_qkv = torch.empty((G, t_local, Hl, 3, hd), dtype=q.dtype, device=dev)
        recv_qkv = torch.empty((t_full, Hl, 3, hd), dtype=q.dtype, device=dev)
        qf, kf_, vf = (torch.empty((t_full, Hl, hd), dtype=q.dtype, device=dev) for _ in range(3))
        of = torch.empty((t_full, Hl, hd), dtype=q.dtype, device=dev)
        lf = torch.empty((t_full, Hl), dtype=torch.float32, device=dev)
        dof = do[:, :Hl].contiguous()
        dqf, dkf, dvf = (torch.empty((t_full, Hl, hd), dtype=q.dtype, device=dev) for _ in range(3))
        send_o = torch.empty((t_full, Hl, hd), dtype=q.dtype, device=dev)
        recv_o = torch.empty((G, t_local, Hl, hd), dtype=q.dtype, device=dev)
        out_local = torch.empty((t_local, H, hd), dtype=q.dtype, device=dev)
        ws_u = torch.empty(api.workspace_size(desc, Hl, hd, q.dtype, api.ZL_OP_BWD), dtype=torch.uint8, device=dev)
        # the all-to-alls are not on this GPU: the receive buffers are filled once from a real pack
        # (a rank-major permutation of actual rows) and keep their content between the calls
        api.ulysses_pack_qkv(G, ql, kl, vl, send_qkv)
        recv_qkv.view(-1).copy_(send_qkv.view(-1))
        api.ulysses_pack_out(G, cu_rank, qf.copy_(q[:, :Hl]), H, send_o)
        recv_o.view(-1).copy_(send_o.view(-1))
        H_report = Hl

        def step():
            api.ulysses_pack_qkv(G, ql, kl, vl, send_qkv)
            api.ulysses_unpack_qkv(G, cu_rank, recv_qkv, H, qf, kf_, vf)
            api.attn_fwd(desc, qf, kf_, vf, w.scale, of, lf, None, None)
            api.attn_bwd(desc, qf, kf_, vf, of, lf, dof, w.scale, dqf, dkf, dvf, ws_u)
            api.ulysses_pack_out(G, cu_rank, of, H, send_o)
            api.ulysses_unpack_out(G, recv_o, H, out_local)
        ulysses_bytes = {
            "pack_qkv": 2 * 3 * t_local * H * hd * 2, "unpack_qkv": 2 * 3 * t_full * Hl * hd * 2,
            "pack_out": 2 * t_full * Hl * hd * 2, "unpack_out": 2 * t_local * H * hd * 2}
    elif args.mode == "gather":
        gdesc = api.SegDesc.of(gathered_descriptor(w))

        def step():
            api.attn_fwd_step(gdesc, q, k, v, w.scale, out, lse, None, None, api.ZL_STEP_FIRST | api.ZL_STEP_LAST)
            api.attn_bwd(gdesc, q, k, v, out, lse, do, w.scale, dq, dk, dv, ws)
    elif args.mode == "ring":
        steps_in = ring_steps(w, q, k, v)
        n_sq = steps_in[0]["n_shard_rows"]
        max_tq = max(st["q"].shape[0] for st in steps_in)
        o_acc = torch.empty((max_tq, H, hd), dtype=torch.float32, device=dev)
        lse_acc = torch.empty((max_tq, H), dtype=torch.float32, device=dev)
        # the backward consumes final outputs in the packed layout; they come from an
        # all-blocks forward made once here (the same values up to rounding)
        api.attn_fwd(desc, q, k, v, w.scale, out, lse, o_part, lse_part)
        if w.num_slots:
            api.lse_merge(desc, o_part, lse_part, out, lse)
        R = len(steps_in)
        bsteps = ring_bwd_steps(w, q, k, v, out, lse, do, dq, dk, dv)
        dq_acc = torch.empty((n_sq, H, hd), dtype=torch.float32, device=dev)

        def step():
            for r, st in enumerate(steps_in):
                flags = (api.ZL_STEP_FIRST if r == 0 else 0) | (api.ZL_STEP_LAST if r == R - 1 else 0)
                api.attn_fwd_step(st["desc"], st["q"], st["k"], st["v"], w.scale, st["out"], st["lse"], o_acc,
                                  lse_acc, flags)
            for b in bsteps:
                api.attn_bwd_step(b["desc"], b["q"], b["k"], b["v"], b["out"], b["lse"], b["do"], w.scale, b["dq"],
                                  b["dk"], b["dv"], dq_acc, b["flags"], ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    api.profile_reset()
    api.profile_enable(True)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        step()
    end.record()
    torch.cuda.synchronize()
    api.profile_enable(False)
    ms = start.elapsed_time(end) / args.steps
    kt = {name: api.profile_read(kid) for kid, name in api.KERNEL_NAMES.items()}
    # per step (a ring step launches the forward once per block)
    avg = {name: (t / args.steps if n else 0.0) for name, (t, n) in kt.items()}

    pairs = w.pair_count()
    if args.mode == "ulysses":
        H = H_report            # this GPU computes H/h heads of every sequence
    fa_flops = 14.0 * hd * H * pairs
    value = fa_flops / (ms * 1e-3) / 1e12
    # MFMA FLOPs per block-diagonal pair (x d x H) each kernel executes (forward S and PV: 4; dK/dV
    # kernel S, dP, dV, dK: 8; dQ kernel S, dP, dQ: 6) and its share of the algorithmic 12 per step
    # (no recompute: the forward's 4, dP, dV and dK of the dK/dV kernel, dQ of the dQ kernel).
    executed = {"fwd": 4.0, "bwd_dkdv": 8.0, "bwd_dq": 6.0}
    algorithmic = {"fwd": 4.0, "bwd_dkdv": 6.0, "bwd_dq": 2.0}
    ceiling = None if args.no_ceiling else gemm_ceiling()
    kern = {}
    for name, f in executed.items():
        if avg.get(name):
            per_s = hd * H * pairs / (avg[name] * 1e-3) / 1e12
            kern[name] = {"ms": round(avg[name], 4),
                          "algorithmic_tflops": round(algorithmic[name] * per_s, 2),
                          "frac": round(algorithmic[name] * per_s / BF16_PEAK_TFLOPS, 4),
                          "executed_tflops": round(f * per_s, 2),
                          "frac_executed": round(f * per_s / BF16_PEAK_TFLOPS, 4),
                          "flops_per_pair_per_d": {"algorithmic": algorithmic[name], "executed": f}}
    dom = max(kern, key=lambda n: kern[n]["ms"])
    alg12 = 12.0 * hd * H * pairs / (ms * 1e-3) / 1e12
    roof = {"bound": "mfma", "kernel": dom, "achieved": kern[dom]["algorithmic_tflops"], "peak": BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": kern[dom]["frac"], "traffic": None,
            "flops_per_pair_per_d": algorithmic[dom],
            "executed_tflops": kern[dom]["executed_tflops"], "frac_executed": kern[dom]["frac_executed"],
            "step_frac_algorithmic_12d": round(alg12 / BF16_PEAK_TFLOPS, 4),
            "step_frac_fa_14d": round(value / BF16_PEAK_TFLOPS, 4)}
    if ceiling:
        roof["measured_ceiling"] = ceiling
        roof["frac_executed_of_measured_ceiling"] = round(kern[dom]["executed_tflops"] / ceiling["tflops"], 4)
    rec = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "mode": args.mode, "heads": H, "head_dim": hd, "total_q": w.total_q,
                   "total_k": w.total_k,
                   "pairs_per_head": pairs, "shard_rows": w.shard_rows(), "num_slots": w.num_slots},
        "pct_of_mfma_peak": round(100.0 * value / BF16_PEAK_TFLOPS, 2),
        "algorithmic_tflops_12d": round(alg12, 2),
        "kernel_ms": {n: round(a, 4) for n, a in avg.items()},
        "kernels": kern,
        "roofline": roof,
    }
    tr = stored_traffic(dom, w.name)
    if tr:
        rec["roofline"]["traffic"] = tr["fetch_bytes"] + tr["write_bytes"]
        rec["roofline"]["traffic_detail"] = {"fetch_bytes": tr["fetch_bytes"], "write_bytes": tr["write_bytes"],
                                             "unique_input_output_bytes": tr.get("unique_bytes")}
    if w.num_slots and avg.get("merge"):
        rec["merge_kernel"] = merge_record(w, H, hd, args.partials, avg["merge"])
        rec["merge_kernel"]["workload"] = w.name
    elif args.mode == "blocks" and args.merge_reps > 0:
        rec["merge_kernel"] = merge_on(args.merge_workload, args.merge_reps, args.partials)
    if "merge_kernel" in rec and not args.no_ceiling:
        cc = hbm_ceilings()
        rec["merge_kernel"]["measured_ceiling"] = cc
        rec["merge_kernel"]["frac_of_measured_read_ceiling"] = round(rec["merge_kernel"]["achieved"] / cc["read_gbs"], 4)
    # Host scheduler: building the forward, dK/dV and dQ work tables of this batch (what the cached
    # plan saves on every later call; zl_plan_dump runs the same builder on the host).
    t0 = time.perf_counter()
    for op in (api.ZL_OP_FWD, api.ZL_OP_BWD, api.ZL_OP_BWD_DQ):
        api.plan_dump(desc, H, hd, q.dtype, op)
    rec["host_scheduler_ms"] = round((time.perf_counter() - t0) * 1e3, 3)
    if args.mode == "blocks" and w.num_slots:
        rec["config"]["partials"] = args.partials
    if args.mode == "ulysses":
        total_b = sum(ulysses_bytes.values())
        ums = avg.get("ulysses", 0.0)
        rec["config"]["ulysses_group"] = args.ulysses_group
        rec["config"]["heads_per_gpu"] = H
        rec["ulysses_staging"] = {"bound": "hbm", "ms": round(ums, 4), "bytes": total_b,
                                  "achieved": round(total_b / (ums * 1e-3) / 1e9, 1) if ums else None,
                                  "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                  "frac": round(total_b / (ums * 1e-3) / 1e9 / HBM_PEAK_GBS, 4) if ums else None,
                                  "bytes_per_call": ulysses_bytes}
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
