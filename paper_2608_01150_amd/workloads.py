"""Synthetic packed whole+shard workloads and their seeded input generator.

This module holds no attention arithmetic: it only describes batches (as
plain integer arrays) and draws their inputs.  Both the GPU path (through
tests and the benchmark) and the fp64 oracle take their inputs from here.

Shapes follow Wan's token arithmetic as the paper uses it (Sec. I: a 15 s
1080p video gives 497,760 tokens): a 480x832 image is 30x52 = 1560 tokens,
a 720x1280 image 45x80 = 3600 tokens, an 81-frame 480x832 video 21 latent
frames x 1560 = 32,760 tokens, a 720p video 21 x 3600 = 75,600 tokens.

Generator.  Every element of every tensor is a pure function of
(seed, tensor id, flat element index), so any slice can be drawn on its own,
on the CPU or on a GPU, with bit-identical values.  The hash is Wellons'
"lowbias32" 32-bit integer mixer (xorshift-multiply, constants 0x7feb352d
and 0x846ca68b), evaluated with int64 arithmetic that never overflows.  Its
32 bits pick a point of the standard normal's quantile function: the top 20
select one of 2^20 equal-probability bins and the low 12 a position inside
it, where the quantile is interpolated linearly between the bin's edges.  The
edge table is computed once per process in fp64 (scipy's ndtri; the two outer
edges are the quantiles at a quarter of a bin from each end), rounded once to
fp32 and shared by every device, and the interpolation is one fp32 multiply
and one add, so CPU and GPU draws agree bit for bit.  The samples follow
N(0,1) to within the curvature of the quantile function inside a bin of
probability 2^-20, tails included, out to about +-5.06 sigma; they are then
rounded once to bf16 (round to nearest even) for bf16 workloads.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Sequence, Tuple

import torch

WHOLE = 0
SHARD = 1

TENSOR_Q, TENSOR_K, TENSOR_V, TENSOR_DO = 0, 1, 2, 3

_M32 = 0xFFFFFFFF


def _mul32(x: torch.Tensor, c: int) -> torch.Tensor:
    """(x * c) mod 2^32 for 0 <= x < 2^32 without int64 overflow."""
    lo, hi = c & 0xFFFF, c >> 16
    return (x * lo + (((x * hi) & 0xFFFF) << 16)) & _M32


def _lowbias32(x: torch.Tensor) -> torch.Tensor:
    x = x ^ (x >> 16)
    x = _mul32(x, 0x7FEB352D)
    x = x ^ (x >> 15)
    x = _mul32(x, 0x846CA68B)
    x = x ^ (x >> 16)
    return x


def _lowbias32_int(x: int) -> int:
    x &= _M32
    x ^= x >> 16
    x = (x * 0x7FEB352D) & _M32
    x ^= x >> 15
    x = (x * 0x846CA68B) & _M32
    x ^= x >> 16
    return x


_QBITS = 20                       # equal-probability bins of the quantile table
_FBITS = 32 - _QBITS              # position inside a bin
_EDGES = {}                       # device -> fp32 bin edges of N(0,1), [2^20 + 1]


def _normal_edges(device) -> torch.Tensor:
    key = str(torch.device(device))
    if key not in _EDGES:
        if "cpu" not in _EDGES:
            import numpy as np
            from scipy.special import ndtri
            n = 1 << _QBITS
            u = np.arange(n + 1, dtype=np.float64) / n
            u[0], u[n] = 0.25 / n, 1.0 - 0.25 / n      # finite outer edges, symmetric
            e = ndtri(u)
            e[n // 2:] = -e[n // 2::-1][:n // 2 + 1]   # exact antisymmetry before rounding
            _EDGES["cpu"] = torch.from_numpy(e.astype(np.float32))
        _EDGES[key] = _EDGES["cpu"].to(device)
    return _EDGES[key]


def draw(seed: int, tensor_id: int, index: torch.Tensor, dtype=torch.bfloat16) -> torch.Tensor:
    """Values at flat element indices ``index`` (int64, < 2^32) of one tensor."""
    k1 = _lowbias32_int(seed * 8 + tensor_id * 2 + 1)
    h = _lowbias32(_lowbias32(index) ^ k1)
    edges = _normal_edges(index.device)
    b = h >> _FBITS
    e0, e1 = edges[b], edges[b + 1]
    w = ((h & ((1 << _FBITS) - 1)) * 2 + 1).to(torch.float32) * (2.0 ** -(_FBITS + 1))   # exact
    step = (e1 - e0) * w            # one rounding
    x = e0 + step                   # one rounding
    return x.to(dtype)


@dataclasses.dataclass(frozen=True)
class Workload:
    """A packed batch: segments, K/V ranges, heads, dtype and seed.

    Field meanings match the C descriptor (``zl_seg_desc``): query segment s
    owns packed rows [cu_seqlens_q[s], cu_seqlens_q[s+1]) and uses K/V ranges
    kv_first[s] .. kv_first[s]+kv_count[s]-1; range j owns packed K/V rows
    [cu_seqlens_k[j], cu_seqlens_k[j+1]) and is CP block block_index[j].
    """
    name: str
    num_heads: int
    head_dim: int
    dtype: str                       # "bf16" or "fp32"
    cu_seqlens_q: Tuple[int, ...]
    kind: Tuple[int, ...]
    q_offset: Tuple[int, ...]
    kv_first: Tuple[int, ...]
    kv_count: Tuple[int, ...]
    cu_seqlens_k: Tuple[int, ...]
    k_offset: Tuple[int, ...]
    block_index: Tuple[int, ...]
    num_slots: int
    seed: int
    scaled_segments: Tuple[int, ...] = ()   # segments whose Q and K are multiplied by 4
    backward: bool = True

    @property
    def total_q(self) -> int:
        return self.cu_seqlens_q[-1]

    @property
    def total_k(self) -> int:
        return self.cu_seqlens_k[-1]

    @property
    def num_segments(self) -> int:
        return len(self.kind)

    @property
    def scale(self) -> float:
        return 1.0 / float(self.head_dim) ** 0.5

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    def pair_count(self) -> int:
        """Sum over (segment, range) of Lq * Lk: the block-diagonal pairs per head."""
        total = 0
        for s in range(self.num_segments):
            lq = self.cu_seqlens_q[s + 1] - self.cu_seqlens_q[s]
            for j in range(self.kv_first[s], self.kv_first[s] + self.kv_count[s]):
                total += lq * (self.cu_seqlens_k[j + 1] - self.cu_seqlens_k[j])
        return total

    def shard_rows(self) -> int:
        return sum(self.cu_seqlens_q[s + 1] - self.cu_seqlens_q[s]
                   for s in range(self.num_segments) if self.kind[s] == SHARD)

    def desc_dict(self) -> dict:
        return {f: getattr(self, f) for f in (
            "cu_seqlens_q", "kind", "q_offset", "kv_first", "kv_count",
            "cu_seqlens_k", "k_offset", "block_index", "num_slots")}

    # -- input generation ---------------------------------------------------
    def _seed_for(self, tensor_id: int) -> int:
        return self.seed

    def rows_of_segment_q(self, s: int) -> Tuple[int, int]:
        return self.cu_seqlens_q[s], self.cu_seqlens_q[s + 1]

    def _q_scale_rows(self):
        return [self.rows_of_segment_q(s) for s in self.scaled_segments]

    def _k_scale_rows(self):
        out = []
        for s in self.scaled_segments:
            for j in range(self.kv_first[s], self.kv_first[s] + self.kv_count[s]):
                out.append((self.cu_seqlens_k[j], self.cu_seqlens_k[j + 1]))
        return out

    def slice(self, tensor_id: int, row0: int, row1: int, heads: Optional[Sequence[int]] = None,
              device="cpu") -> torch.Tensor:
        """Rows [row0, row1) of one input tensor, shape [rows, len(heads), d]."""
        h_all, d = self.num_heads, self.head_dim
        heads = list(range(h_all)) if heads is None else list(heads)
        t = torch.arange(row0, row1, dtype=torch.int64, device=device)
        hh = torch.tensor(heads, dtype=torch.int64, device=device)
        c = torch.arange(d, dtype=torch.int64, device=device)
        idx = ((t[:, None, None] * h_all + hh[None, :, None]) * d + c[None, None, :])
        x = draw(self.seed, tensor_id, idx, self.torch_dtype)
        scaled = (self._q_scale_rows() if tensor_id == TENSOR_Q
                  else self._k_scale_rows() if tensor_id == TENSOR_K else [])
        for a, b in scaled:
            lo, hi = max(a, row0), min(b, row1)
            if lo < hi:
                x[lo - row0:hi - row0] *= 4   # exact in bf16 and fp32
        return x

    def full(self, tensor_id: int, device="cpu", chunk_rows: int = 65536) -> torch.Tensor:
        rows = self.total_q if tensor_id in (TENSOR_Q, TENSOR_DO) else self.total_k
        out = torch.empty((rows, self.num_heads, self.head_dim), dtype=self.torch_dtype, device=device)
        for r0 in range(0, rows, chunk_rows):
            r1 = min(rows, r0 + chunk_rows)
            out[r0:r1] = self.slice(tensor_id, r0, r1, device=device)
        return out


def _build(name, H, d, dtype, segments, seed, scaled=(), backward=True, block_order=None):
    """segments: list of ("whole", L, q_offset) or ("shard", Lq, q_offset, [(Lk, k_offset, block)]).

    Whole segments get their own K/V range; shard segments list their blocks.
    A block given as an int refers to an earlier shard's range index (shared
    K/V), which only forward-only workloads use.
    """
    cq, ck = [0], [0]
    kind, qoff, first, count, koff, bidx = [], [], [], [], [], []
    for seg in segments:
        if seg[0] == "whole":
            _, length, off = seg
            kind.append(WHOLE)
            qoff.append(off)
            cq.append(cq[-1] + length)
            first.append(len(ck) - 1)
            count.append(1)
            ck.append(ck[-1] + length)
            koff.append(off)
            bidx.append(0)
        else:
            _, lq, off, blocks = seg
            kind.append(SHARD)
            qoff.append(off)
            cq.append(cq[-1] + lq)
            if isinstance(blocks, tuple) and blocks and blocks[0] == "shared":
                first.append(blocks[1])
                count.append(blocks[2])
                continue
            first.append(len(ck) - 1)
            count.append(len(blocks))
            for (lk, ko, b) in blocks:
                ck.append(ck[-1] + lk)
                koff.append(ko)
                bidx.append(b)
    used = [bidx[j] for s in range(len(kind)) if kind[s] == SHARD
            for j in range(first[s], first[s] + count[s])]
    nslots = 1 + max(used) if used else 0
    return Workload(name=name, num_heads=H, head_dim=d, dtype=dtype,
                    cu_seqlens_q=tuple(cq), kind=tuple(kind), q_offset=tuple(qoff),
                    kv_first=tuple(first), kv_count=tuple(count), cu_seqlens_k=tuple(ck),
                    k_offset=tuple(koff), block_index=tuple(bidx), num_slots=nslots,
                    seed=seed, scaled_segments=tuple(scaled), backward=backward)


def seeded_choice(seed: int, n: int) -> int:
    """First index of a seeded permutation of range(n) (hash order)."""
    keys = [(_lowbias32_int(_lowbias32_int(seed) ^ i), i) for i in range(n)]
    return min(keys)[1]


def tiny_plumbing() -> Workload:
    """fp32 forward-only plumbing case: whole 64/128/256 plus one 256-token
    sequence split into four 64-query shards that each attend to all four
    64-token K/V blocks (the blocks are shared by the four shards)."""
    segs = [("whole", 64, 0), ("whole", 128, 0), ("whole", 256, 0),
            ("shard", 64, 0, [(64, 0, 0), (64, 64, 1), (64, 128, 2), (64, 192, 3)])]
    for i in (1, 2, 3):
        segs.append(("shard", 64, 64 * i, ("shared", 3, 4)))
    return _build("tiny-plumbing-fp32", 2, 64, "fp32", segs, 20260001, backward=False)


def image_only() -> Workload:
    """16 whole 1560-token images, 12 heads, d=128, bf16."""
    return _build("image-16x1560-h12", 12, 128, "bf16",
                  [("whole", 1560, 0)] * 16, 20260002)


def mixed_image_video() -> Workload:
    """One 32,760-token video, two 3600-token and eight 1560-token images,
    40 heads, d=128, bf16; one seeded segment (10% of 11, rounded) has Q and
    K scaled by 4 to stress the softmax range."""
    segs = [("whole", 32760, 0)] + [("whole", 3600, 0)] * 2 + [("whole", 1560, 0)] * 8
    scaled = (seeded_choice(20260103, len(segs)),)
    return _build("mixed-video32760+2x3600+8x1560-h40", 40, 128, "bf16", segs, 20260003, scaled)


def coalesced_shard(cp=8, shard=9450, fillers=(1560,) * 6) -> Workload:
    """One GPU's share of a 75,600-token 720p video at CP=8 (a 9450-query
    shard against all 8 K/V blocks, merged) packed with six whole 1560-token
    images in the same launch, 40 heads, d=128, bf16.  The shard comes first
    (the engine orders segments by decreasing split degree)."""
    blocks = [(shard, b * shard, b) for b in range(cp)]
    segs = [("shard", shard, 0, blocks)] + [("whole", L, 0) for L in fillers]
    return _build(f"coalesced-shard{shard}x{cp}+{len(fillers)}fill-h40", 40, 128, "bf16", segs, 20260004)


def long_video_shard() -> Workload:
    """One GPU's share of a 497,760-token 1080p video at CP=16 (31,110
    queries against 16 blocks of 31,110) with four 3600-token and eight
    1560-token whole fillers, 40 heads, d=128, bf16."""
    w = coalesced_shard(cp=16, shard=31110, fillers=(3600,) * 4 + (1560,) * 8)
    return dataclasses.replace(w, name="long-shard31110x16+12fill-h40", seed=20260005)


# -- bucket catalog and synthetic batches (for the price table) -----------------
# Wan2.1 latent geometry: 8x spatial VAE compression with 2x2 patches gives
# (H/16) x (W/16) tokens per latent frame; 4x temporal compression of a
# 16 fps clip of F = 16*seconds + 1 frames gives 1 + (F-1)/4 latent frames.
# Frame sizes: 256p = 256x448, 480p = 480x832, 720p = 720x1280, 1080p =
# 1088x1920 (the height padded to a multiple of 16, which reproduces the
# 497,760 tokens of a 15 s 1080p video in Sec. I).
_FRAME = {"256p": (256, 448), "480p": (480, 832), "720p": (720, 1280), "1080p": (1088, 1920)}


def tokens_per_frame(res: str) -> int:
    h, w = _FRAME[res]
    return (h // 16) * (w // 16)


def latent_frames(seconds: int, fps: int = 16) -> int:
    return 1 + (fps * seconds) // 4


def _catalog():
    cat = {f"img{r[:-1]}": tokens_per_frame(r) for r in _FRAME}
    for sec in (5, 10, 15):
        for r in ("480p", "720p", "1080p"):
            cat[f"vid{r[:-1]}-{sec}s"] = latent_frames(sec) * tokens_per_frame(r)
    return cat


CATALOG = _catalog()       # bucket name -> whole-sequence tokens
IMAGE_BUCKETS = tuple(b for b in CATALOG if b.startswith("img"))


def synthetic_batch(num_ranks: int, tokens_per_rank: int, video_share: float, seconds: int, seed: int):
    """A seeded mixed image-video batch in the shape of the paper's suites
    (Sec. V-A: 480p-1080p videos of one duration, 256p-1080p images, a
    per-GPU token budget and a video-token share).  Videos of uniformly drawn
    resolution are added while the video tokens stay within the share (at
    least one video), then images of uniformly drawn resolution until the
    budget is reached.  Returns bucket names, videos first."""
    import random
    rng = random.Random(seed)
    total = num_ranks * tokens_per_rank
    vids = [f"vid{r}-{seconds}s" for r in ("480", "720", "1080")]
    out, vt = [], 0
    while True:
        b = rng.choice(vids)
        if out and vt + CATALOG[b] > video_share * total:
            break
        out.append(b)
        vt += CATALOG[b]
    t = vt
    while True:
        b = rng.choice(IMAGE_BUCKETS)
        if t + CATALOG[b] > total:
            break
        out.append(b)
        t += CATALOG[b]
    return out


def build_segments(name: str, H: int, d: int, segments, seed: int) -> Workload:
    """A bf16 fwd+bwd workload from a segment list: ("whole", L, q_offset) or
    ("shard", Lq, q_offset, [(Lk, k_offset, block), ...])."""
    return _build(name, H, d, "bf16", segments, seed)


WORKLOADS = {
    "c1": tiny_plumbing,
    "c2": image_only,
    "c3": mixed_image_video,
    "c4": coalesced_shard,
    "c5": long_video_shard,
}


def get(name: str) -> Workload:
    return WORKLOADS[name]()
