"""Pins for the oracle's forward (attention of one key range, packed batches).

Each pin checks the oracle against something other than itself: 50-digit
decimal brute force, closed forms, and invariants of exact attention.
"""
import math

import numpy as np
import pytest

import oracle
from tests._decimal_ref import attend_decimal


@pytest.mark.parametrize("lq,lk,d", [(1, 1, 1), (3, 5, 4), (8, 8, 4), (5, 2, 3), (7, 8, 2)])
def test_forward_matches_decimal_brute_force(rng, lq, lk, d):
    q, k, v = (rng.standard_normal((n, d)) * 2 for n in (lq, lk, lk))
    scale = 0.7
    o, lse = oracle.attend(q, k, v, scale)
    od, lsed = attend_decimal(q.tolist(), k.tolist(), v.tolist(), scale)
    for i in range(lq):
        assert abs(float(lsed[i]) - lse[i]) <= 1e-14 * max(1.0, abs(lse[i]))
        for c in range(d):
            assert abs(float(od[i][c]) - o[i, c]) <= 1e-14 * max(1.0, abs(o[i, c]))


def test_single_key_closed_form(rng):
    q, k, v = rng.standard_normal((4, 6)), rng.standard_normal((1, 6)), rng.standard_normal((1, 6))
    o, lse = oracle.attend(q, k, v, 0.3)
    np.testing.assert_allclose(o, np.repeat(v, 4, axis=0), rtol=0, atol=1e-15)
    np.testing.assert_allclose(lse, 0.3 * (q @ k[0]), rtol=1e-15, atol=1e-15)


def test_two_keys_closed_form(rng):
    q, k, v = rng.standard_normal((5, 3)), rng.standard_normal((2, 3)), rng.standard_normal((2, 3))
    scale = 1.3
    o, lse = oracle.attend(q, k, v, scale)
    for i in range(5):
        s1, s2 = scale * q[i] @ k[0], scale * q[i] @ k[1]
        w1 = 1.0 / (1.0 + math.exp(s2 - s1))  # logistic sigma(s1 - s2)
        w2 = 1.0 / (1.0 + math.exp(s1 - s2))
        np.testing.assert_allclose(o[i], w1 * v[0] + w2 * v[1], rtol=1e-13, atol=1e-14)
        hi = max(s1, s2)
        assert abs(lse[i] - (hi + math.log1p(math.exp(-abs(s1 - s2))))) < 1e-13


def test_zero_queries_give_mean_and_log_count(rng):
    k, v = rng.standard_normal((9, 4)), rng.standard_normal((9, 4))
    o, lse = oracle.attend(np.zeros((3, 4)), k, v, 0.5)
    np.testing.assert_allclose(o, np.tile(v.mean(axis=0), (3, 1)), rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(lse, np.full(3, math.log(9)), rtol=1e-15)


def test_constant_v_returns_that_row(rng):
    q, k = rng.standard_normal((6, 8)) * 3, rng.standard_normal((11, 8)) * 3
    row = rng.standard_normal(8)
    o, _ = oracle.attend(q, k, np.tile(row, (11, 1)), 0.9)
    np.testing.assert_allclose(o, np.tile(row, (6, 1)), rtol=1e-13, atol=1e-14)


def test_key_permutation_invariance(rng):
    q, k, v = rng.standard_normal((5, 4)), rng.standard_normal((13, 4)), rng.standard_normal((13, 4))
    perm = rng.permutation(13)
    o1, l1 = oracle.attend(q, k, v, 0.8)
    o2, l2 = oracle.attend(q, k[perm], v[perm], 0.8)
    np.testing.assert_allclose(o1, o2, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(l1, l2, rtol=1e-14, atol=1e-14)


def test_key_shift_moves_lse_only(rng):
    q, k, v = rng.standard_normal((5, 4)), rng.standard_normal((7, 4)), rng.standard_normal((7, 4))
    u = rng.standard_normal(4)
    o1, l1 = oracle.attend(q, k, v, 0.6)
    o2, l2 = oracle.attend(q, k + u, v, 0.6)
    np.testing.assert_allclose(o1, o2, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(l2, l1 + 0.6 * (q @ u), rtol=1e-13, atol=1e-13)


def test_large_logits_stay_finite(rng):
    # Logits near 100 (the x4-scaled segments reach ~70): max-subtraction keeps it exact.
    q = rng.standard_normal((4, 16)) * 8
    k = rng.standard_normal((6, 16)) * 8
    v = rng.standard_normal((6, 16))
    o, lse = oracle.attend(q, k, v, 0.25)
    od, lsed = attend_decimal(q.tolist(), k.tolist(), v.tolist(), 0.25)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    np.testing.assert_allclose(lse, [float(x) for x in lsed], rtol=1e-14)
    np.testing.assert_allclose(o, [[float(x) for x in r] for r in od], rtol=1e-12, atol=1e-14)


def test_empty_key_range():
    o, lse = oracle.attend(np.ones((3, 4)), np.zeros((0, 4)), np.zeros((0, 4)), 1.0)
    assert np.all(o == 0) and np.all(lse == -np.inf)


def _tiny_desc():
    # whole 5, whole 3, shard 4 queries vs blocks of 3 and 6 keys (slots 1 and 0)
    return dict(cu_seqlens_q=(0, 5, 8, 12), kind=(0, 0, 1), q_offset=(0, 0, 2),
                kv_first=(0, 1, 2), kv_count=(1, 1, 2), cu_seqlens_k=(0, 5, 8, 11, 17),
                k_offset=(0, 0, 0, 3), block_index=(0, 0, 1, 0), num_slots=2)


def test_packed_forward_routes_segments_and_slots(rng):
    desc = _tiny_desc()
    H, d = 2, 4
    q, k, v = rng.standard_normal((12, H, d)), rng.standard_normal((17, H, d)), rng.standard_normal((17, H, d))
    r = oracle.packed_forward(desc, q, k, v, 0.5)
    for h in range(H):
        o, lse = oracle.attend(q[0:5, h], k[0:5, h], v[0:5, h], 0.5)
        np.testing.assert_array_equal(r["out"][0:5, h], o)
        o, lse = oracle.attend(q[5:8, h], k[5:8, h], v[5:8, h], 0.5)
        np.testing.assert_array_equal(r["lse"][5:8, h], lse)
        o, lse = oracle.attend(q[8:12, h], k[8:11, h], v[8:11, h], 0.5)
        np.testing.assert_array_equal(r["o_part"][1, 8:12, h], o)
        o, lse = oracle.attend(q[8:12, h], k[11:17, h], v[11:17, h], 0.5)
        np.testing.assert_array_equal(r["lse_part"][0, 8:12, h], lse)
    # shard rows never written to out, whole rows never to the partials
    assert np.all(np.isnan(r["out"][8:12])) and np.all(np.isnan(r["o_part"][:, 0:8]))


def test_packed_segment_isolation(rng):
    """Block-diagonal attention keeps sequences separate (Sec. IV-D)."""
    desc = _tiny_desc()
    q, k, v = rng.standard_normal((12, 1, 4)), rng.standard_normal((17, 1, 4)), rng.standard_normal((17, 1, 4))
    a = oracle.packed_forward(desc, q, k, v, 0.5)
    k2, v2, q2 = k.copy(), v.copy(), q.copy()
    k2[5:8] += 10.0
    v2[5:8] -= 3.0
    q2[5:8] *= -2
    b = oracle.packed_forward(desc, q2, k2, v2, 0.5)
    for key in ("out", "lse", "final_out", "final_lse"):
        np.testing.assert_array_equal(a[key][0:5], b[key][0:5])
        np.testing.assert_array_equal(a[key][8:12], b[key][8:12])
        assert not np.allclose(a[key][5:8], b[key][5:8])
