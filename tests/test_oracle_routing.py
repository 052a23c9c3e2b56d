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


# ---------------------------------------------------------------------------
# Tie-break order, written out by hand.  The rule: cost = q_len * k_len
# descending, then (segment, head, q_start, k_start, range) ascending.  The
# descriptor below makes many items cost the same, with the tie keys
# disagreeing in every way the packing allows:
#   ranges  r0 [0, 64)  r1 [64, 192)  r2 [192, 256)  r3 [256, 320)  r4 [320, 352)
#   seg 0   WHOLE rows [0, 128)    on r1
#   seg 1   SHARD rows [128, 256)  on r2 (slot 1), r3 (slot 0)
#   seg 2   SHARD rows [256, 320)  on r0 (slot 0)   (a later segment on an earlier range)
#   seg 3   WHOLE rows [320, 352)  on r4
# Tiles: 64 query rows (forward, dQ), 64 keys (dK/dV).  Each list below was
# derived on paper from the rule, item by item; it is not produced by any
# sort key.  Items are (q_start, q_len, k_start, k_len, head, slot, segment,
# range).
# ---------------------------------------------------------------------------
TIE = dict(cu_seqlens_q=(0, 128, 256, 320, 352), kind=(0, 1, 1, 0), q_offset=(0, 0, 0, 0),
           kv_first=(1, 2, 0, 4), kv_count=(1, 2, 1, 1), cu_seqlens_k=(0, 64, 192, 256, 320, 352),
           k_offset=(0, 0, 0, 64, 0), block_index=(0, 0, 1, 0, 0), num_slots=2)

TIE_FWD = [
    # cost 64*128: seg 0, head 0 before head 1, query tiles in order
    (0, 64, 64, 128, 0, -1, 0, 1), (64, 64, 64, 128, 0, -1, 0, 1),
    (0, 64, 64, 128, 1, -1, 0, 1), (64, 64, 64, 128, 1, -1, 0, 1),
    # cost 64*64: seg 1 before seg 2 (although seg 2's keys come first); within
    # seg 1 head, then query tile, then block
    (128, 64, 192, 64, 0, 1, 1, 2), (128, 64, 256, 64, 0, 0, 1, 3),
    (192, 64, 192, 64, 0, 1, 1, 2), (192, 64, 256, 64, 0, 0, 1, 3),
    (128, 64, 192, 64, 1, 1, 1, 2), (128, 64, 256, 64, 1, 0, 1, 3),
    (192, 64, 192, 64, 1, 1, 1, 2), (192, 64, 256, 64, 1, 0, 1, 3),
    (256, 64, 0, 64, 0, 0, 2, 0), (256, 64, 0, 64, 1, 0, 2, 0),
    # cost 32*32
    (320, 32, 320, 32, 0, -1, 3, 4), (320, 32, 320, 32, 1, -1, 3, 4),
]

TIE_BWD = [
    # cost 128*64: seg 0 (two key tiles of r1) before seg 1 (one tile each of r2, r3)
    (0, 128, 64, 64, 0, -1, 0, 1), (0, 128, 128, 64, 0, -1, 0, 1),
    (0, 128, 64, 64, 1, -1, 0, 1), (0, 128, 128, 64, 1, -1, 0, 1),
    (128, 128, 192, 64, 0, 1, 1, 2), (128, 128, 256, 64, 0, 0, 1, 3),
    (128, 128, 192, 64, 1, 1, 1, 2), (128, 128, 256, 64, 1, 0, 1, 3),
    # cost 64*64, then 32*32
    (256, 64, 0, 64, 0, 0, 2, 0), (256, 64, 0, 64, 1, 0, 2, 0),
    (320, 32, 320, 32, 0, -1, 3, 4), (320, 32, 320, 32, 1, -1, 3, 4),
]

TIE_DQ = [
    # cost 64*128: seg 0 (its 128 keys), then seg 1 (r2 and r3 together, 128 keys from row 192)
    (0, 64, 64, 128, 0, -1, 0, 1), (64, 64, 64, 128, 0, -1, 0, 1),
    (0, 64, 64, 128, 1, -1, 0, 1), (64, 64, 64, 128, 1, -1, 0, 1),
    (128, 64, 192, 128, 0, -1, 1, 2), (192, 64, 192, 128, 0, -1, 1, 2),
    (128, 64, 192, 128, 1, -1, 1, 2), (192, 64, 192, 128, 1, -1, 1, 2),
    (256, 64, 0, 64, 0, -1, 2, 0), (256, 64, 0, 64, 1, -1, 2, 0),
    (320, 32, 320, 32, 0, -1, 3, 4), (320, 32, 320, 32, 1, -1, 3, 4),
]


@pytest.mark.parametrize("op,expect", [(0, TIE_FWD), (1, TIE_BWD), (2, TIE_DQ)])
def test_tie_break_order_written_by_hand(op, expect):
    assert oracle.work_items(TIE, 2, op, 64, 64) == expect


# Field positions in an item tuple.
_QS, _QL, _KS, _KL, _HD, _SG, _RG = 0, 1, 2, 3, 4, 6, 7


@pytest.mark.parametrize("a,b", [(x, y) for i, x in enumerate("shqkr") for y in "shqkr"[i + 1:]])
def test_swapped_tie_keys_fail_the_hand_lists(a, b):
    """Discriminating power of the pins above: re-sorting the same items with two tie keys swapped
    reproduces none of the hand lists, except for swapping k_start and range, which cannot be told
    apart: a segment's ranges are consecutive and their rows never decrease, so within one
    (segment, head, q_start) the two keys always agree."""
    pos = {"s": _SG, "h": _HD, "q": _QS, "k": _KS, "r": _RG}
    keys = list("shqkr")
    i, j = keys.index(a), keys.index(b)
    keys[i], keys[j] = keys[j], keys[i]
    differs = []
    for expect in (TIE_FWD, TIE_BWD, TIE_DQ):
        mutant = sorted(expect, key=lambda it: (-(it[_QL] * it[_KL]),) + tuple(it[pos[c]] for c in keys))
        differs.append(mutant != expect)
    if {a, b} == {"k", "r"}:
        assert not any(differs)
    else:
        assert any(differs), f"swapping {a} and {b} goes unnoticed"
