"""The library's schedule (zl_plan_dump) against the oracle's independent
derivation: the same work items in the same order, bit for bit."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_01150_amd import api
from paper_2608_01150_amd import workloads as W
from tests import _descs


def _compare(d, H, hd, dtype, op):
    items, (tm, tn) = api.plan_dump(api.SegDesc.of(d), H, hd, dtype, op)
    ref = np.array(oracle.work_items(d, H, op, tm, tn), dtype=np.int32).reshape(-1, 8)
    assert items.shape == ref.shape
    np.testing.assert_array_equal(items, ref)
    return items, tm, tn


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5"])
def test_workload_schedules_match_oracle(name):
    w = W.get(name)
    ops = [api.ZL_OP_FWD] + ([api.ZL_OP_BWD, api.ZL_OP_BWD_DQ] if w.backward else [])
    for op in ops:
        items, tm, tn = _compare(w.desc_dict() | {"q_offset": w.q_offset, "k_offset": w.k_offset},
                                 w.num_heads, w.head_dim, w.torch_dtype, op)
        # every (row, head, range) pair is covered: total work equals the pair count
        assert int((items[:, 1].astype(np.int64) * items[:, 3]).sum()) == w.pair_count() * w.num_heads


def test_random_descriptor_schedules_match_oracle():
    rng = np.random.default_rng(7)
    for trial in range(25):
        d = _descs.random_desc(rng, int(rng.integers(0, 5)), int(rng.integers(0, 4)), 300, 5)
        if not d["kind"]:
            continue
        for op in (api.ZL_OP_FWD, api.ZL_OP_BWD, api.ZL_OP_BWD_DQ):
            for dtype in (torch.bfloat16, torch.float32):
                if op != api.ZL_OP_FWD and dtype == torch.float32:
                    continue
                _compare(d, int(rng.integers(1, 4)), 64, dtype, op)


def test_schedule_is_deterministic():
    d = api.SegDesc.of(_descs.mixed_small())
    a, _ = api.plan_dump(d, 3, 128, torch.bfloat16, api.ZL_OP_FWD)
    b, _ = api.plan_dump(d, 3, 128, torch.bfloat16, api.ZL_OP_FWD)
    np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("name", ["c3", "c4"])
def test_list_schedule_bound(name):
    """Greedy list scheduling of the issue order on m workgroup slots finishes
    within Graham's bound total/m + (1 - 1/m) * max_item, and the LPT order
    keeps the tail short: makespan / (total/m) stays near 1."""
    import heapq
    w = W.get(name)
    items, _ = api.plan_dump(api.SegDesc.of(w), w.num_heads, w.head_dim, w.torch_dtype, api.ZL_OP_FWD)
    cost = items[:, 1].astype(np.float64) * items[:, 3]
    m = 512  # 256 CUs x 2 resident workgroups
    heap = [0.0] * m
    for c in cost:
        t = heapq.heappop(heap)
        heapq.heappush(heap, t + c)
    makespan = max(heap)
    total = cost.sum()
    assert makespan <= total / m + (1 - 1 / m) * cost.max() + 1e-6
    assert makespan / (total / m) < 1.05


def test_zero_row_shard_keeps_its_key_tiles():
    """A SHARD segment without query rows has no forward or dQ work, but its blocks' dK/dV are outputs
    of the backward (zero), so the dK/dV schedule still covers them: key tiles of 128 with q_len 0,
    ordered after every item of positive cost."""
    d = _descs.desc(cu_q=(0, 100, 100), kind=(0, 1), kv_first=(0, 1), kv_count=(1, 2),
                    cu_k=(0, 100, 300, 430), block_index=(0, 1, 0), num_slots=2)
    items, (tm, tn) = api.plan_dump(api.SegDesc.of(d), 1, 128, torch.bfloat16, api.ZL_OP_BWD)
    assert tn == 128
    want = [(0, 100, 0, 100, 0, -1, 0, 0),
            (100, 0, 100, 128, 0, 1, 1, 1), (100, 0, 228, 72, 0, 1, 1, 1),
            (100, 0, 300, 128, 0, 0, 1, 2), (100, 0, 428, 2, 0, 0, 1, 2)]
    assert [tuple(int(x) for x in it) for it in items] == want
    for op in (api.ZL_OP_FWD, api.ZL_OP_BWD_DQ):
        items, _ = api.plan_dump(api.SegDesc.of(d), 1, 128, torch.bfloat16, op)
        assert set(items[:, 6].tolist()) == {0}
