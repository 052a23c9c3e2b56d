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


# ---------------------------------------------------------------------------
# attend_bwd_given: the backward on a supplied (stored) O and LSE.
# ---------------------------------------------------------------------------

def test_given_exact_o_lse_is_the_backward(rng):
    q, k, v, do = (rng.standard_normal((n, 5)) for n in (7, 11, 11, 7))
    o, lse = oracle.attend(q, k, v, 0.7)
    for a, b in zip(oracle.attend_bwd_given(q, k, v, do, o, lse, 0.7), oracle.attend_bwd(q, k, v, do, 0.7)):
        np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-13)


def test_given_lse_shift_equals_scaled_upstream_gradient(rng):
    """LSE_i + eps_i multiplies every P_ij of row i by exp(-eps_i), so the gradients equal those of the
    exact backward (pinned by finite differences above) with dO_i scaled by exp(-eps_i)."""
    q, k, v, do = (rng.standard_normal((n, 4)) for n in (6, 9, 9, 6))
    o, lse = oracle.attend(q, k, v, 0.5)
    eps = rng.uniform(-2.0, 2.0, size=6)
    got = oracle.attend_bwd_given(q, k, v, do, o, lse + eps, 0.5)
    want = oracle.attend_bwd(q, k, v, do * np.exp(-eps)[:, None], 0.5)
    for a, b in zip(got, want):
        np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-13)


def test_given_perturbed_o_moves_only_d_brute_force(rng):
    """O_i + delta_i changes only D_i, by dO_i . delta_i; dS_ij then moves by -P_ij dO_i . delta_i.
    The expected change is evaluated entry by entry with math.exp (brute force on a tiny case)."""
    import math
    lq, lk, d, sc = 4, 5, 3, 0.9
    q, k, v, do = (rng.standard_normal((n, d)) for n in (lq, lk, lk, lq))
    o, lse = oracle.attend(q, k, v, sc)
    delta = 1e-2 * rng.standard_normal((lq, d))
    base = oracle.attend_bwd_given(q, k, v, do, o, lse, sc)
    moved = oracle.attend_bwd_given(q, k, v, do, o + delta, lse, sc)
    ddq, ddk = np.zeros((lq, d)), np.zeros((lk, d))
    for i in range(lq):
        dd = sum(do[i, c] * delta[i, c] for c in range(d))
        for j in range(lk):
            p = math.exp(sc * sum(q[i, c] * k[j, c] for c in range(d)) - lse[i])
            for c in range(d):
                ddq[i, c] -= sc * p * dd * k[j, c]
                ddk[j, c] -= sc * p * dd * q[i, c]
    np.testing.assert_allclose(moved[0] - base[0], ddq, rtol=1e-9, atol=1e-13)
    np.testing.assert_allclose(moved[1] - base[1], ddk, rtol=1e-9, atol=1e-13)
    np.testing.assert_array_equal(moved[2], base[2])  # dV does not read D


def test_given_row_subsets(rng):
    q, k, v, do = (rng.standard_normal((n, 4)) for n in (9, 13, 13, 9))
    o, lse = oracle.attend(q, k, v, 0.6)
    full = oracle.attend_bwd_given(q, k, v, do, o, lse, 0.6)
    rows = np.array([1, 4, 8])
    sub_q, _, _ = oracle.attend_bwd_given(q[rows], k, v, do[rows], o[rows], lse[rows], 0.6,
                                          k_rows=np.array([], dtype=np.int64))
    np.testing.assert_allclose(sub_q, full[0][rows], rtol=1e-13, atol=1e-14)
