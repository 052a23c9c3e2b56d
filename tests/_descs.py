"""Small hand-made descriptors shared by CPU and GPU tests (plain data)."""
import numpy as np


def desc(cu_q, kind, kv_first, kv_count, cu_k, block_index, num_slots, q_offset=None, k_offset=None):
    return dict(cu_seqlens_q=tuple(cu_q), kind=tuple(kind), kv_first=tuple(kv_first), kv_count=tuple(kv_count),
                cu_seqlens_k=tuple(cu_k), block_index=tuple(block_index), num_slots=num_slots,
                q_offset=None if q_offset is None else tuple(q_offset),
                k_offset=None if k_offset is None else tuple(k_offset))


def mixed_small():
    """whole 200, empty whole, whole 77, a 150-query shard vs blocks of 300/0/129
    keys (slots 2, 0, 1), a 33-query shard vs one 64-key block (slot 0)."""
    return desc(cu_q=(0, 200, 200, 277, 427, 460), kind=(0, 0, 0, 1, 1),
                kv_first=(0, 1, 2, 3, 6), kv_count=(1, 1, 1, 3, 1),
                cu_k=(0, 200, 200, 277, 577, 577, 706, 770), block_index=(0, 0, 0, 2, 0, 1, 0),
                num_slots=3, q_offset=(0, 0, 0, 0, 500), k_offset=(0, 0, 0, 0, 300, 300, 500))


def random_desc(rng, n_whole, n_shard, max_len, max_blocks, allow_empty=True):
    cu_q, cu_k, kind, first, count, bidx = [0], [0], [], [], [], []
    kinds = [0] * n_whole + [1] * n_shard
    rng.shuffle(kinds)
    nslots = 0
    lo = 0 if allow_empty else 1
    for kd in kinds:
        lq = int(rng.integers(lo, max_len + 1))
        cu_q.append(cu_q[-1] + lq)
        kind.append(kd)
        first.append(len(cu_k) - 1)
        if kd == 0:
            count.append(1)
            cu_k.append(cu_k[-1] + lq)
            bidx.append(0)
        else:
            nb = int(rng.integers(1, max_blocks + 1))
            count.append(nb)
            slots = rng.permutation(max_blocks)[:nb]
            for b in slots:
                cu_k.append(cu_k[-1] + int(rng.integers(lo, max_len + 1)))
                bidx.append(int(b))
            nslots = max(nslots, max_blocks)
    return desc(cu_q, kind, first, count, cu_k, bidx, nslots)
