"""Pins for the oracle's backward: central finite differences of the loss
L = sum(dO * O), closed-form column sums, and the shard/whole equivalence."""
import numpy as np
import pytest

import oracle


def _loss(q, k, v, do, scale):
    o, _ = oracle.attend(q, k, v, scale)
    return float((do * o).sum())


@pytest.mark.parametrize("lq,lk,d", [(1, 1, 2), (3, 4, 3), (5, 7, 4), (6, 2, 5)])
def test_backward_matches_finite_differences(rng, lq, lk, d):
    q, k, v = rng.standard_normal((lq, d)), rng.standard_normal((lk, d)), rng.standard_normal((lk, d))
    do = rng.standard_normal((lq, d))
    scale, h = 0.8, 1e-6
    dq, dk, dv = oracle.attend_bwd(q, k, v, do, scale)
    for x, g in ((q, dq), (k, dk), (v, dv)):
        num = np.zeros_like(x)
        for idx in np.ndindex(*x.shape):
            old = x[idx]
            x[idx] = old + h
            lp = _loss(q, k, v, do, scale)
            x[idx] = old - h
            lm = _loss(q, k, v, do, scale)
            x[idx] = old
            num[idx] = (lp - lm) / (2 * h)
        err = np.abs(num - g).max() / max(1.0, np.abs(g).max())
        assert err <= 1e-6, err


def test_column_sums_closed_form(rng):
    # sum_j dS_ij = 0 for every row, hence sum_j dK_j = 0; sum_j P_ij = 1, hence sum_j dV_j = sum_i dO_i.
    q, k, v, do = (rng.standard_normal((n, 6)) for n in (9, 12, 12, 9))
    dq, dk, dv = oracle.attend_bwd(q, k, v, do, 0.4)
    np.testing.assert_allclose(dk.sum(axis=0), 0.0, atol=1e-13)
    np.testing.assert_allclose(dv.sum(axis=0), do.sum(axis=0), rtol=1e-13, atol=1e-13)


def test_row_and_key_subsets_match_full(rng):
    q, k, v, do = (rng.standard_normal((n, 4)) for n in (10, 15, 15, 10))
    dq, dk, dv = oracle.attend_bwd(q, k, v, do, 0.5)
    rows, keys = np.array([0, 3, 9]), np.array([14, 2, 7, 8])
    sq, sk, sv = oracle.attend_bwd(q, k, v, do, 0.5, q_rows=rows, k_rows=keys)
    np.testing.assert_allclose(sq, dq[rows], rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(sk, dk[keys], rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(sv, dv[keys], rtol=1e-13, atol=1e-14)


def test_shards_sum_to_whole_gradients(rng):
    """A 12-token sequence kept whole vs split into three 4-query shards that
    each attend to the sequence's three 4-key blocks: the gradients of every
    query row and of every key row agree (exactness of CP, Sec. II-B)."""
    H, d = 2, 3
    q, k, v, do = (rng.standard_normal((12, H, d)) for _ in range(4))
    whole = dict(cu_seqlens_q=(0, 12), kind=(0,), q_offset=(0,), kv_first=(0,), kv_count=(1,),
                 cu_seqlens_k=(0, 12), k_offset=(0,), block_index=(0,), num_slots=0)
    shard = dict(cu_seqlens_q=(0, 4, 8, 12), kind=(1, 1, 1), q_offset=(0, 4, 8),
                 kv_first=(0, 0, 0), kv_count=(3, 3, 3), cu_seqlens_k=(0, 4, 8, 12),
                 k_offset=(0, 4, 8), block_index=(0, 1, 2), num_slots=3)
    gw = oracle.packed_backward(whole, q, k, v, do, 0.6)
    gs = oracle.packed_backward(shard, q, k, v, do, 0.6)
    for a, b in zip(gw, gs):
        np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-13)
