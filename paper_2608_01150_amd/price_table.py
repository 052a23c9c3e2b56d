"""Single-GPU price table and a check of the additive load model.

The planner of arXiv 2608.01150 prices every (catalog bucket, parallelism
configuration) pair once per training setup (Sec. IV-B, the Hardware
Profiler): the per-participating-rank time P_{b,theta}, and a rank's load is
the sum of the prices of what it runs.  On one GPU the part of a price that
can be measured is the local attention compute (forward and backward) a
rank performs for its share, so that is what this table holds; the
collectives are not run (one GPU).

Configurations, each priced for rank 0's share (even splits, the first
shares one row longer):
  whole        (1,1,1): the sequence alone.  Buckets shorter than
               2^17 tokens are priced inside a packed launch of n copies
               (time / n), as the engine coalesces whole sequences.
  ring-k       (1,1,k): L/k queries against the k blocks of the sequence in
               one coalesced launch, their partials LSE-merged.
  gather-q     (q,1,1): L/q queries against the gathered L keys, one range.
  ulysses-h    (1,h,1): the QKV pack/unpack, all L tokens on H/h heads, the
               output pack/unpack (h must divide H).

``check`` then plans a synthetic batch with the table: videos are anchors,
each split with ring-g over an aligned group of g ranks (a fixed greedy
stand-in for the CP-SAT anchor stage); images are fillers placed by
zl_fill_pack (Eq. 8).  Each rank's
coalesced launch (its anchor shards and its fillers) is then run and timed
and compared with the predicted load, the local-compute analogue of the
additive-model evaluation of Sec. V-B.

Usage:
  python -m paper_2608_01150_amd.price_table measure --heads 12 --out prices.json
  python -m paper_2608_01150_amd.price_table check --prices prices.json
"""
from __future__ import annotations

import argparse
import json
import sys
import time

import numpy as np
import torch

from . import api
from . import workloads as W

PACK_TOKENS = 1 << 17


def even_split(n: int, parts: int):
    """Lengths of `parts` even shards of n (the first n % parts one longer)."""
    return [n // parts + (1 if j < n % parts else 0) for j in range(parts)]


def config_segments(L: int, config: str):
    """Segment list of rank 0's local work for one sequence of L tokens."""
    kind, _, deg = config.partition("-")
    if kind == "whole":
        return [("whole", L, 0)]
    k = int(deg)
    shard = even_split(L, k)
    if kind == "ring":
        offs = np.concatenate([[0], np.cumsum(shard)]).tolist()
        return [("shard", shard[0], 0, [(shard[b], offs[b], b) for b in range(k)])]
    if kind == "gather":
        return [("shard", shard[0], 0, [(L, 0, 0)])]
    if kind == "ulysses":
        return [("whole", L, 0)]
    raise ValueError(config)


class Runner:
    """Inputs and outputs of one workload resident on the GPU, and one
    fwd+bwd pass of it through the library."""

    def __init__(self, w: W.Workload, mode: str, dev, ulysses_group: int = 1, full_heads: int = 0):
        self.w, self.mode, self.dev = w, mode, dev
        H, d = w.num_heads, w.head_dim
        self.desc = api.SegDesc.of(w)
        self.q = w.full(W.TENSOR_Q, device=dev)
        self.k = w.full(W.TENSOR_K, device=dev)
        self.v = w.full(W.TENSOR_V, device=dev)
        self.do = w.full(W.TENSOR_DO, device=dev)
        self.out = torch.empty_like(self.q)
        self.lse = torch.empty((w.total_q, H), dtype=torch.float32, device=dev)
        self.o_part = self.lse_part = None
        if mode == "blocks" and w.num_slots:
            self.o_part = torch.empty((w.num_slots, w.total_q, H, d), dtype=torch.float32, device=dev)
            self.lse_part = torch.empty((w.num_slots, w.total_q, H), dtype=torch.float32, device=dev)
        self.dq, self.dk, self.dv = torch.empty_like(self.q), torch.empty_like(self.k), torch.empty_like(self.v)
        self.ws = torch.empty(api.workspace_size(self.desc, H, d, self.q.dtype, api.ZL_OP_BWD), dtype=torch.uint8,
                              device=dev)
        self.group = ulysses_group
        if mode == "ulysses":
            G, Hf = ulysses_group, full_heads
            L = w.total_q
            self.cu_rank = np.array([[0, n] for n in even_split(L, G)], np.int32)
            t_local = int(self.cu_rank[0][1])
            src = W.build_segments("ulysses-local", Hf, d, [("whole", t_local, 0)], w.seed + 1)
            self.ql = src.full(W.TENSOR_Q, device=dev)
            self.kl = src.full(W.TENSOR_K, device=dev)
            self.vl = src.full(W.TENSOR_V, device=dev)
            self.send_qkv = torch.empty((G, t_local, H, 3, d), dtype=self.q.dtype, device=dev)
            api.ulysses_pack_qkv(G, self.ql, self.kl, self.vl, self.send_qkv)
            self.recv_qkv = torch.zeros((L, H, 3, d), dtype=self.q.dtype, device=dev)
            n = min(self.recv_qkv.numel(), self.send_qkv.numel())
            self.recv_qkv.view(-1)[:n].copy_(self.send_qkv.view(-1)[:n])
            self.send_o = torch.empty((L, H, d), dtype=self.q.dtype, device=dev)
            self.recv_o = torch.zeros((G, t_local, H, d), dtype=self.q.dtype, device=dev)
            self.out_local = torch.empty((t_local, Hf, d), dtype=self.q.dtype, device=dev)
            self.full_heads = Hf

    def step(self):
        w = self.w
        if self.mode == "ulysses":
            G = self.group
            api.ulysses_pack_qkv(G, self.ql, self.kl, self.vl, self.send_qkv)
            api.ulysses_unpack_qkv(G, self.cu_rank, self.recv_qkv, self.full_heads, self.q, self.k, self.v)
        if self.mode == "gather":
            api.attn_fwd_step(self.desc, self.q, self.k, self.v, w.scale, self.out, self.lse, None, None,
                              api.ZL_STEP_FIRST | api.ZL_STEP_LAST)
        else:
            api.attn_fwd(self.desc, self.q, self.k, self.v, w.scale, self.out, self.lse, self.o_part, self.lse_part)
            if self.o_part is not None:
                api.lse_merge(self.desc, self.o_part, self.lse_part, self.out, self.lse)
        api.attn_bwd(self.desc, self.q, self.k, self.v, self.out, self.lse, self.do, w.scale, self.dq, self.dk,
                     self.dv, self.ws)
        if self.mode == "ulysses":
            api.ulysses_pack_out(self.group, self.cu_rank, self.out, self.full_heads, self.send_o)
            api.ulysses_unpack_out(self.group, self.recv_o, self.full_heads, self.out_local)

    def time_ms(self, budget_s: float = 10.0) -> float:
        """Median over timed passes after one warm-up pass; fewer passes for
        long ones so a whole table stays within minutes."""
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        self.step()
        ev[1].record()
        torch.cuda.synchronize()
        first = ev[0].elapsed_time(ev[1])
        reps = int(max(2, min(7, budget_s * 1e3 / max(first, 1e-3) / 3)))
        ts = []
        for _ in range(reps):
            ev[0].record()
            self.step()
            ev[1].record()
            torch.cuda.synchronize()
            ts.append(ev[0].elapsed_time(ev[1]))
        return float(np.median(ts))


def price_one(bucket: str, config: str, H: int, d: int, dev, seed: int = 20260100):
    L = W.CATALOG[bucket]
    kind, _, deg = config.partition("-")
    copies = 1
    if kind == "whole" and L < PACK_TOKENS:
        copies = max(1, PACK_TOKENS // L)
    segs = config_segments(L, config) * copies
    if kind == "ulysses":
        h = int(deg)
        w = W.build_segments(f"{bucket}-{config}", H // h, d, segs, seed)
        r = Runner(w, "ulysses", dev, ulysses_group=h, full_heads=H)
    else:
        w = W.build_segments(f"{bucket}-{config}", H, d, segs, seed)
        r = Runner(w, "gather" if kind == "gather" else "blocks", dev)
    ms = r.time_ms() / copies
    del r
    torch.cuda.empty_cache()
    return ms, copies


def configs_for(bucket: str, H: int, degrees):
    out = ["whole"]
    if bucket.startswith("vid"):
        for k in degrees:
            out += [f"ring-{k}", f"gather-{k}"]
            if H % k == 0:
                out.append(f"ulysses-{k}")
    return out


def measure(args):
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    degrees = [int(x) for x in args.degrees.split(",")]
    buckets = args.buckets.split(",") if args.buckets else list(W.CATALOG)
    table = {"heads": args.heads, "head_dim": args.head_dim, "dtype": "bf16", "unit": "ms",
             "what": "local attention fwd+bwd time of rank 0's share, one MI355X", "prices": {}}
    t0 = time.time()
    for b in buckets:
        table["prices"][b] = {"tokens": W.CATALOG[b]}
        for c in configs_for(b, args.heads, degrees):
            ms, copies = price_one(b, c, args.heads, args.head_dim, dev)
            table["prices"][b][c] = round(ms, 5)
            print(f"[price] {b:12s} {c:11s} {ms:10.4f} ms" + (f"  (packed x{copies})" if copies > 1 else "")
                  + f"  t={time.time() - t0:.0f}s", flush=True)
    with open(args.out, "w") as f:
        json.dump(table, f, indent=1)
    print(json.dumps({"price_table": args.out, "seconds": round(time.time() - t0, 1)}), flush=True)


# -- plan a synthetic batch with the table and check the additive model ---------------

def plan(batch, prices, num_ranks: int, anchor_degree: int, bytes_per_token: float, mem_cap: float,
         filler_rule: str):
    """Anchors (videos) split with ring-g over aligned groups of g ranks,
    most expensive first, each to the group whose busiest rank is least loaded
    (a fixed stand-in for the CP-SAT anchor stage; g = 1 keeps them whole).
    Fillers (images) then go by Eq. 8 (filler_rule "eq8") or, for
    comparison, to the rank with the fewest tokens so far ("tokens").
    Returns the anchor placement [(bucket, first rank)], per-rank filler
    lists, the predicted load ledger, the memory ledger and F."""
    N, g = num_ranks, anchor_degree
    if N % g:
        raise ValueError("the anchor degree must divide the number of ranks")
    P = prices["prices"]
    cfg = "whole" if g == 1 else f"ring-{g}"
    anchors = [b for b in batch if b.startswith("vid")]
    fillers = [b for b in batch if not b.startswith("vid")]
    load = [0.0] * N
    mem = [0.0] * N
    placed = []
    for b in sorted(anchors, key=lambda b: -P[b][cfg]):
        first = min(range(0, N, g), key=lambda f: max(load[f:f + g]))
        for j in range(g):
            load[first + j] += P[b][cfg]
            mem[first + j] += even_split(W.CATALOG[b], g)[j] * bytes_per_token
        placed.append((b, first))
    floor = sum(P[b]["whole"] for b in batch) / N
    if filler_rule == "eq8":
        price = [P[b]["whole"] for b in fillers]
        need = np.array([[W.CATALOG[b] * bytes_per_token] * N for b in fillers]).reshape(len(fillers), N)
        rank_of, load, mem, failed = api.fill_pack(price, need, load, mem, floor, mem_cap)
        if failed is not None:
            raise RuntimeError(f"filler packing failed at filler {failed}")
        rank_of = rank_of.tolist()
        load, mem = load.tolist(), mem.tolist()
    else:
        tok = [0] * N
        for b, first in placed:
            for j in range(g):
                tok[first + j] += even_split(W.CATALOG[b], g)[j]
        rank_of = []
        for b in fillers:
            r = int(np.argmin(tok))
            rank_of.append(r)
            tok[r] += W.CATALOG[b]
            load[r] += P[b]["whole"]
            mem[r] += W.CATALOG[b] * bytes_per_token
    per_rank = [[fillers[i] for i in range(len(fillers)) if rank_of[i] == r] for r in range(N)]
    return placed, per_rank, load, mem, floor


def rank_segments(placed, fillers, g: int, r: int):
    """Rank r's coalesced segment list: its anchor shards (ring-g, all g
    blocks each) first, as the engine orders by decreasing split degree, then
    its whole fillers."""
    segs = []
    for b, first in placed:
        if not first <= r < first + g:
            continue
        L = W.CATALOG[b]
        if g == 1:
            segs.append(("whole", L, 0))
            continue
        sh = even_split(L, g)
        offs = np.concatenate([[0], np.cumsum(sh)]).tolist()
        j = r - first
        segs.append(("shard", sh[j], offs[j], [(sh[i], offs[i], i) for i in range(g)]))
    for b in fillers:
        segs.append(("whole", W.CATALOG[b], 0))
    return segs


def check(args):
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    prices = json.load(open(args.prices))
    H, d = prices["heads"], prices["head_dim"]
    N = args.ranks
    batch = W.synthetic_batch(N, args.tokens_per_rank, args.video_share, args.seconds, args.seed)
    report = {"ranks": N, "anchor_degree": args.anchor_degree, "tokens_per_rank": args.tokens_per_rank, "video_share": args.video_share,
              "seconds": args.seconds, "seed": args.seed, "heads": H, "batch": {}, "plans": {}}
    for b in batch:
        report["batch"][b] = report["batch"].get(b, 0) + 1
    for rule in args.rules.split(","):
        placed, per_rank, load, mem, floor = plan(batch, prices, N, args.anchor_degree, args.bytes_per_token,
                                                  args.mem_cap_gib * 2 ** 30, rule)
        meas = []
        for r in range(N):
            w = W.build_segments(f"rank{r}", H, d, rank_segments(placed, per_rank[r], args.anchor_degree, r),
                                 args.seed + r)
            run = Runner(w, "blocks", dev)
            ms = run.time_ms(budget_s=8.0)
            del run
            torch.cuda.empty_cache()
            meas.append(ms)
            print(f"[check] {rule:6s} rank {r}: {len(per_rank[r]):3d} fillers, predicted {load[r]:9.3f} ms, "
                  f"measured {ms:9.3f} ms", flush=True)
        err = [abs(m - p) / m for m, p in zip(meas, load)]
        report["plans"][rule] = {
            "predicted_ms": [round(x, 3) for x in load], "measured_ms": [round(x, 3) for x in meas],
            "fillers_per_rank": [len(x) for x in per_rank], "load_floor_ms": round(floor, 3),
            "anchor_first_rank": [[b, f] for b, f in placed],
            "mape": round(float(np.mean(err)), 4), "max_ape": round(float(np.max(err)), 4),
            "predicted_makespan_ms": round(max(load), 3), "measured_makespan_ms": round(max(meas), 3),
            "measured_imbalance": round(max(meas) / float(np.mean(meas)), 4),
            "memory_gib": [round(x / 2 ** 30, 2) for x in mem]}
    with open(args.out, "w") as f:
        json.dump(report, f, indent=1)
    print(json.dumps({k: v for k, v in report.items() if k != "batch"}), flush=True)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    m = sub.add_parser("measure")
    m.add_argument("--heads", type=int, default=12)
    m.add_argument("--head-dim", type=int, default=128)
    m.add_argument("--degrees", default="2,4,8,16")
    m.add_argument("--buckets", default="", help="comma-separated subset of the catalog (default: all)")
    m.add_argument("--out", required=True)
    c = sub.add_parser("check")
    c.add_argument("--prices", required=True)
    c.add_argument("--ranks", type=int, default=8)
    c.add_argument("--tokens-per-rank", type=int, default=350_000)
    c.add_argument("--video-share", type=float, default=0.5)
    c.add_argument("--seconds", type=int, default=10)
    c.add_argument("--seed", type=int, default=20260200)
    c.add_argument("--anchor-degree", type=int, default=4, help="ring degree g of every anchor (1 = whole)")
    c.add_argument("--bytes-per-token", type=float, default=150e3)
    c.add_argument("--mem-cap-gib", type=float, default=220.0)
    c.add_argument("--rules", default="eq8,tokens")
    c.add_argument("--out", required=True)
    args = ap.parse_args(argv)
    if not torch.cuda.is_available():
        print("price_table needs a GPU: it times the library's kernels", file=sys.stderr)
        return 2
    (measure if args.cmd == "measure" else check)(args)
    return 0


if __name__ == "__main__":
    sys.exit(main())
