"""Pins for the oracle's routing and work-item derivation."""
import collections

import pytest

import oracle

DESC = dict(cu_seqlens_q=(0, 300, 300, 364, 428), kind=(0, 0, 1, 1), q_offset=(0, 0, 0, 64),
            kv_first=(0, 1, 2, 2), kv_count=(1, 1, 3, 3), cu_seqlens_k=(0, 300, 300, 364, 364, 492),
            k_offset=(0, 0, 0, 64, 64), block_index=(0, 0, 2, 0, 1), num_slots=3)


def test_row_routing():
    rows = oracle.row_routing(DESC)
    assert len(rows) == 428
    assert rows[0] == (0, 0, 0, ()) and rows[299] == (0, 0, 299, ())
    assert rows[300] == (2, 1, 0, (2, 0, 1))
    assert rows[427] == (3, 1, 64 + 63, (2, 0, 1))


@pytest.mark.parametrize("op,bm,bn", [(0, 128, 64), (0, 64, 64), (1, 128, 128), (1, 64, 32)])
def test_items_cover_every_pair_once(op, bm, bn):
    H = 3
    items = oracle.work_items(DESC, H, op, bm, bn)
    cover = collections.Counter()
    for (q0, ql, k0, kl, h, slot, s, j) in items:
        assert (ql <= bm) if op == 0 else (kl <= bn)
        for r in range(q0, q0 + ql):
            cover[(r, h, j)] += kl if kl else 1
    expect = collections.Counter()
    for s in range(4):
        for r in range(DESC["cu_seqlens_q"][s], DESC["cu_seqlens_q"][s + 1]):
            for j in range(DESC["kv_first"][s], DESC["kv_first"][s] + DESC["kv_count"][s]):
                lk = DESC["cu_seqlens_k"][j + 1] - DESC["cu_seqlens_k"][j]
                if op == 1 and lk == 0:
                    continue
                for h in range(H):
                    expect[(r, h, j)] += lk if lk else 1
    assert cover == expect
    costs = [it[1] * it[3] for it in items]
    assert costs == sorted(costs, reverse=True)


def test_dq_items_cover_each_row_once_with_all_keys():
    items = oracle.work_items(DESC, 2, 2, 128, 64)
    rows = collections.Counter()
    for (q0, ql, k0, kl, h, slot, s, j) in items:
        assert slot == -1 and j == DESC["kv_first"][s]
        first, count = DESC["kv_first"][s], DESC["kv_count"][s]
        ck = DESC["cu_seqlens_k"]
        assert kl == ck[first + count] - ck[first] and k0 == ck[first]
        for r in range(q0, q0 + ql):
            rows[(r, h)] += 1
    assert rows == collections.Counter({(r, h): 1 for r in range(428) for h in range(2)})


def test_slots_follow_block_index():
    for (q0, ql, k0, kl, h, slot, s, j) in oracle.work_items(DESC, 1, 0, 128, 64):
        assert slot == (DESC["block_index"][j] if DESC["kind"][s] == 1 else -1)
