"""Seeded mutation fuzzing of descriptor validation and scheduling, on the host
only: zl_plan_dump validates a descriptor and builds its schedule without a
GPU, so no kernel is ever launched here.

Each trial takes a valid random descriptor (with or without global offsets),
changes one to three values to edge cases, and requires that
  * the library either accepts it or rejects it with ZL_ERR_INVALID_ARG and a
    message, never another status or a crash;
  * it accepts exactly the descriptors that the rules stated in zl_attn.h
    accept (written out again below from the header, not from the library);
  * an accepted descriptor's forward and backward schedules equal the
    oracle's derivation, item for item.
Counts (num_q_segs, num_kv_ranges) are never mutated: they size the host
arrays the library reads.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_01150_amd import api
from tests import _descs

OFF_MAX = 2**63 - 1 - 2**31
I32_MAX = 2**31 - 1


def with_offsets(d, rng):
    """The descriptor with consistent global offsets: each WHOLE segment and its
    range share one position; the blocks of a SHARD tile disjoint positions."""
    d = dict(d)
    nq = len(d["kind"])
    ck = d["cu_seqlens_k"]
    k_off = [0] * (len(ck) - 1)
    q_off = [0] * nq
    base = int(rng.integers(0, 1000))
    for s in range(nq):
        f, c = d["kv_first"][s], d["kv_count"][s]
        if d["kind"][s] == 0:
            q_off[s] = k_off[f] = base
            base += ck[f + 1] - ck[f] + 7
        else:
            q_off[s] = base
            for j in range(f, f + c):
                k_off[j] = base
                base += ck[j + 1] - ck[j] + 3
    d["q_offset"], d["k_offset"] = tuple(q_off), tuple(k_off)
    return d


def header_accepts(d):
    """The validity rules of zl_seg_desc as zl_attn.h states them."""
    cq, ck = d["cu_seqlens_q"], d["cu_seqlens_k"]
    kind, first, count, bidx = d["kind"], d["kv_first"], d["kv_count"], d["block_index"]
    qo, ko, ns = d["q_offset"], d["k_offset"], d["num_slots"]
    nq, nk = len(kind), len(ck) - 1
    if cq[0] != 0 or ck[0] != 0 or ns < 0:
        return False
    if any(cq[i + 1] < cq[i] for i in range(nq)) or any(ck[j + 1] < ck[j] for j in range(nk)):
        return False
    if ko is not None and any(not 0 <= x <= OFF_MAX for x in ko):
        return False
    if qo is not None and any(not 0 <= x <= OFF_MAX for x in qo):
        return False
    for s in range(nq):
        f, c = first[s], count[s]
        if kind[s] not in (0, 1) or c < 1 or f < 0 or f + c > nk:
            return False
        lq = cq[s + 1] - cq[s]
        if kind[s] == 0:
            if c != 1 or ck[f + 1] - ck[f] != lq:
                return False
            if qo is not None and ko is not None and qo[s] != ko[f]:
                return False
        else:
            slots = [bidx[j] for j in range(f, f + c)]
            if any(not 0 <= b < ns for b in slots) or len(set(slots)) != len(slots):
                return False
            if ko is not None:
                # blocks cover [k_offset, k_offset + length); an empty block covers no token
                spans = [(ko[j], ko[j] + ck[j + 1] - ck[j]) for j in range(f, f + c) if ck[j + 1] > ck[j]]
                if any(a0 < b1 and b0 < a1 for i, (a0, a1) in enumerate(spans) for (b0, b1) in spans[:i]):
                    return False
    return True


def mutate(d, rng):
    d = {k: (list(v) if isinstance(v, tuple) else v) for k, v in d.items()}
    nq, nk = len(d["kind"]), len(d["cu_seqlens_k"]) - 1
    field = rng.choice(["cu_seqlens_q", "cu_seqlens_k", "kind", "kv_first", "kv_count", "block_index", "num_slots",
                        "q_offset", "k_offset"])
    if field == "num_slots":
        d["num_slots"] = int(rng.choice([-1, 0, 1, d["num_slots"] + 1, max(d["num_slots"] - 1, 0)]))
        return d
    arr = d[field]
    if arr is None or len(arr) == 0:
        return d
    i = int(rng.integers(0, len(arr)))
    cur = arr[i]
    if field in ("cu_seqlens_q", "cu_seqlens_k"):
        cands = [0, -1, cur - 1, cur + 1, cur + 64, max(cur - 64, 0)]
    elif field == "kind":
        cands = [0, 1, 2, 255]
    elif field == "kv_first":
        cands = [-1, 0, nk - 1, nk, cur + 1, I32_MAX]
    elif field == "kv_count":
        cands = [-1, 0, 1, 2, nk, cur + 1, I32_MAX]
    elif field == "block_index":
        cands = [-1, 0, d["num_slots"] - 1, d["num_slots"], arr[max(i - 1, 0)]]
    else:
        cands = [-1, 0, cur + 1, cur - 1, OFF_MAX, OFF_MAX + 1, 2**63 - 1, -(2**63)]
    arr[i] = int(rng.choice(cands))
    return d


def _status(d, op):
    sd = api.SegDesc.of(d)
    n = api.ctypes.c_size_t(0)
    st = api._plan_dump(sd.ptr(), 2, 64, api._dtype_code(torch.bfloat16), op, None, 0, api.ctypes.byref(n), None, None)
    return st


@pytest.mark.parametrize("seed", range(4))
def test_mutated_descriptors_follow_the_header_rules(seed):
    rng = np.random.default_rng(20261200 + seed)
    checked = accepted = 0
    for trial in range(150):
        d = _descs.random_desc(rng, int(rng.integers(0, 4)), int(rng.integers(1, 4)), 200, 4)
        if rng.random() < 0.5:
            d = with_offsets(d, rng)
        assert header_accepts(d) and _status(d, api.ZL_OP_FWD) == api.ZL_OK
        for _ in range(int(rng.integers(1, 4))):
            d = mutate(d, rng)
        d = {k: (tuple(v) if isinstance(v, list) else v) for k, v in d.items()}
        want = header_accepts(d)
        st = _status(d, api.ZL_OP_FWD)
        if want:
            assert st == api.ZL_OK, (d, api.last_error())
            accepted += 1
            for op in (api.ZL_OP_FWD, api.ZL_OP_BWD, api.ZL_OP_BWD_DQ):
                items, (tm, tn) = api.plan_dump(api.SegDesc.of(d), 2, 64, torch.bfloat16, op)
                ref = np.array(oracle.work_items(d, 2, op, tm, tn), dtype=np.int32).reshape(-1, 8)
                np.testing.assert_array_equal(items, ref)
        else:
            assert st == api.ZL_ERR_INVALID_ARG, (d, st)
            assert api.last_error()
        checked += 1
    # both outcomes are exercised
    assert 0 < accepted < checked


def test_empty_block_inside_another_is_accepted():
    """An empty block covers no global token, so its offset may lie inside a
    sibling block; a non-empty block there is an overlap."""
    d = _descs.desc(cu_q=(0, 8), kind=(1,), kv_first=(0,), kv_count=(2,), cu_k=(0, 16, 16), block_index=(0, 1),
                    num_slots=2, q_offset=(0,), k_offset=(100, 105))
    assert header_accepts(d) and _status(d, api.ZL_OP_FWD) == api.ZL_OK
    d = _descs.desc(cu_q=(0, 8), kind=(1,), kv_first=(0,), kv_count=(2,), cu_k=(0, 16, 17), block_index=(0, 1),
                    num_slots=2, q_offset=(0,), k_offset=(100, 105))
    assert not header_accepts(d)
    assert _status(d, api.ZL_OP_FWD) == api.ZL_ERR_INVALID_ARG and "overlap" in api.last_error()
