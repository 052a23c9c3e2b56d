"""Pins for the oracle's LSE merge: merging the per-block partials of a shard
must equal exact attention over the concatenated blocks (ring attention keeps
K/V blocks sharded and accumulates the output, Sec. II-B and Tab. II)."""
import math

import numpy as np
import pytest

import oracle


@pytest.mark.parametrize("sizes", [(3,), (4, 4, 4, 4), (1, 7, 2), (5, 0, 6), (2, 9, 1, 3, 8)])
def test_merge_of_blocks_equals_whole(rng, sizes):
    d, lq = 4, 6
    q = rng.standard_normal((lq, d)) * 2
    ks = [rng.standard_normal((n, d)) * 2 for n in sizes]
    vs = [rng.standard_normal((n, d)) for n in sizes]
    parts = [oracle.attend(q, k, v, 0.7) for k, v in zip(ks, vs)]
    o, lse = oracle.lse_merge(np.stack([p[0] for p in parts]), np.stack([p[1] for p in parts]))
    ow, lw = oracle.attend(q, np.concatenate(ks), np.concatenate(vs), 0.7)
    np.testing.assert_allclose(o, ow, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, lw, rtol=1e-12, atol=1e-12)


def test_two_slot_closed_form():
    o1, o2 = np.array([[1.0, 2.0]]), np.array([[-3.0, 0.5]])
    a, b = 0.25, 1.75
    o, lse = oracle.lse_merge(np.stack([o1, o2]), np.array([[a], [b]]))
    den = math.exp(a) + math.exp(b)
    np.testing.assert_allclose(o[0], (math.exp(a) * o1[0] + math.exp(b) * o2[0]) / den, rtol=1e-15)
    assert abs(lse[0] - math.log(den)) < 1e-15


def test_single_slot_is_identity(rng):
    o1, l1 = rng.standard_normal((1, 5, 3)), rng.standard_normal((1, 5))
    o, lse = oracle.lse_merge(o1, l1)
    np.testing.assert_allclose(o, o1[0], rtol=1e-15)
    np.testing.assert_allclose(lse, l1[0], rtol=1e-15)


def test_minus_inf_slots(rng):
    o_parts = rng.standard_normal((3, 4, 2))
    lse_parts = rng.standard_normal((3, 4))
    lse_parts[1, :] = -np.inf          # an empty block everywhere
    lse_parts[:, 3] = -np.inf          # a row with no keys at all
    o, lse = oracle.lse_merge(o_parts, lse_parts)
    ref, lref = oracle.lse_merge(o_parts[[0, 2], :3], lse_parts[[0, 2], :3])
    np.testing.assert_allclose(o[:3], ref, rtol=1e-15)
    np.testing.assert_allclose(lse[:3], lref, rtol=1e-15)
    assert np.all(o[3] == 0) and lse[3] == -np.inf


def test_packed_final_equals_merge_of_slots(rng):
    desc = dict(cu_seqlens_q=(0, 4, 10), kind=(0, 1), q_offset=(0, 4),
                kv_first=(0, 1), kv_count=(1, 3), cu_seqlens_k=(0, 4, 7, 7, 12),
                k_offset=(0, 0, 3, 3), block_index=(0, 2, 0, 1), num_slots=3)
    q, k, v = rng.standard_normal((10, 2, 4)), rng.standard_normal((12, 2, 4)), rng.standard_normal((12, 2, 4))
    r = oracle.packed_forward(desc, q, k, v, 0.5)
    for h in range(2):
        o, lse = oracle.lse_merge(r["o_part"][:, 4:10, h], r["lse_part"][:, 4:10, h])
        np.testing.assert_allclose(o, r["final_out"][4:10, h], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(lse, r["final_lse"][4:10, h], rtol=1e-12, atol=1e-12)
    # slot 0 is the empty range: O_b = 0, LSE_b = -inf
    assert np.all(r["lse_part"][0, 4:10] == -np.inf) and np.all(r["o_part"][0, 4:10] == 0)
