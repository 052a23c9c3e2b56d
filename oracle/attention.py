"""fp64 definitions of exact non-causal attention, its LSE merge and backward.

TEST INFRASTRUCTURE (see the package docstring): never called by the product.

What the paper fixes (arXiv 2608.01150):
  * Sec. II-A: DiT self-attention is dense over all L^2 token pairs of a
    sequence (no causal mask).
  * Sec. II-B and Tab. II: context parallelism exchanges K/V so that each
    rank computes *exact* attention for its query shard; the ring primitive
    keeps K/V blocks sharded and accumulates the output over the blocks.
  * Sec. IV-D: whole sequences of a rank are packed into one block-diagonal
    attention call that keeps sequences separate and returns outputs in the
    rank-local input order; configuration (1,1,1) (Sec. IV-A) keeps a
    sequence whole.
The paper never writes the attention formulas; the ones below are the plain
definitions of softmax attention with a log-sum-exp (LSE) statistic, which is
what its cited FlashAttention and ring-attention executors compute.

Readings where the paper is silent (each is listed in the design notes):
  * LSE is natural-log, includes the softmax scale, fp32 on the GPU.
  * A shard's per-block partial is the block-locally normalised output
    O_b = softmax_b(S) V_b together with LSE_b; exp(LSE_b) * O_b is the raw
    numerator, so the merge is the same either way.
  * An empty key block gives O_b = 0, LSE_b = -inf; the merge ignores -inf
    slots; all slots -inf gives O = 0, LSE = -inf.
  * The shard backward uses the final (merged) O and LSE over all of the
    sequence's keys; dQ of a shard row sums over its blocks.
"""
from __future__ import annotations

import numpy as np

WHOLE = 0
SHARD = 1

# Query rows processed per step.  Every quantity below is defined row by row
# (a query row's LSE and output depend on that row only), so taking the rows
# a block at a time selects rows; it does not reassociate any sum.
_ROW_BLOCK = 2048


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def attend(q, k, v, scale):
    """Exact softmax attention of query rows over one key/value range.

    q [Lq, d], k [Lk, d], v [Lk, d]; returns (O [Lq, d], LSE [Lq]) in fp64 with
      S_ij  = scale * q_i . k_j
      LSE_i = m_i + ln sum_j exp(S_ij - m_i),   m_i = max_j S_ij
      O_i   = sum_j exp(S_ij - LSE_i) v_j
    Lk == 0 gives O = 0 and LSE = -inf (the empty-block reading).
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    lq, d = q.shape
    lk = k.shape[0]
    o = np.zeros((lq, v.shape[1]), np.float64)
    lse = np.full(lq, -np.inf, np.float64)
    if lk == 0 or lq == 0:
        return o, lse
    for r0 in range(0, lq, _ROW_BLOCK):
        r1 = min(lq, r0 + _ROW_BLOCK)
        s = scale * (q[r0:r1] @ k.T)
        m = s.max(axis=1)
        lse[r0:r1] = m + np.log(np.exp(s - m[:, None]).sum(axis=1))
        p = np.exp(s - lse[r0:r1, None])
        o[r0:r1] = p @ v
    return o, lse


def lse_merge(o_parts, lse_parts):
    """Combine per-block partials of the same query rows into exact attention.

    o_parts [B, L, d] (block-locally normalised), lse_parts [B, L]:
      M   = max_b LSE_b
      LSE = M + ln sum_b exp(LSE_b - M)
      O   = sum_b exp(LSE_b - LSE) O_b
    Slots with LSE_b = -inf contribute nothing; if every slot is -inf the row
    is O = 0, LSE = -inf.
    """
    o_parts, lse_parts = _f64(o_parts), _f64(lse_parts)
    nb, length = lse_parts.shape
    o = np.zeros(o_parts.shape[1:], np.float64)
    lse = np.full(length, -np.inf, np.float64)
    if nb == 0:
        return o, lse
    m = lse_parts.max(axis=0)
    live = np.isfinite(m)
    if not live.any():
        return o, lse
    ml = m[live]
    w_un = np.exp(lse_parts[:, live] - ml[None, :])  # exp(-inf) = 0
    lse[live] = ml + np.log(w_un.sum(axis=0))
    w = np.exp(lse_parts[:, live] - lse[live][None, :])
    o[live] = np.einsum("bl,bld->ld", w, o_parts[:, live])
    return o, lse


def attend_bwd(q, k, v, do, scale, q_rows=None, k_rows=None):
    """Gradients of exact attention, from the definitions.

    With (O, LSE) = attend(q, k, v, scale) and upstream gradient dO:
      D_i   = dO_i . O_i
      P_ij  = exp(S_ij - LSE_i)
      dV_j  = sum_i P_ij dO_i
      dP_ij = dO_i . v_j
      dS_ij = P_ij (dP_ij - D_i)
      dQ_i  = scale * sum_j dS_ij k_j
      dK_j  = scale * sum_i dS_ij q_i
    ``q_rows`` / ``k_rows`` (index arrays, default all) select which dQ rows
    and which dK/dV rows are returned, so a large segment can be checked on a
    sample; the selected rows are computed exactly as in the full case.
    Returns (dq [len(q_rows), d], dk [len(k_rows), d], dv [len(k_rows), d]).
    """
    q, k, v, do = _f64(q), _f64(k), _f64(v), _f64(do)
    lq, lk = q.shape[0], k.shape[0]
    qi = np.arange(lq) if q_rows is None else np.asarray(q_rows, np.int64)
    kj = np.arange(lk) if k_rows is None else np.asarray(k_rows, np.int64)
    dq = np.zeros((qi.size, k.shape[1]), np.float64)
    dk = np.zeros((kj.size, q.shape[1]), np.float64)
    dv = np.zeros((kj.size, do.shape[1]), np.float64)
    if lq == 0 or lk == 0:
        return dq, dk, dv
    # O and LSE are row-local: only the rows the requested gradients read
    # are evaluated (every row when any dK/dV row is requested).
    need = np.arange(lq) if kj.size else qi
    o = np.zeros((lq, v.shape[1]), np.float64)
    lse = np.zeros(lq, np.float64)
    o[need], lse[need] = attend(q[need], k, v, scale)
    dsum = (do * o).sum(axis=1)  # D_i

    # dQ for the selected query rows: needs every key of those rows.
    if qi.size:
        s = scale * (q[qi] @ k.T)
        p = np.exp(s - lse[qi, None])
        dp = do[qi] @ v.T
        ds = p * (dp - dsum[qi, None])
        dq = scale * (ds @ k)

    # dK, dV for the selected keys: needs every query of those key columns.
    if kj.size:
        s = scale * (q @ k[kj].T)
        p = np.exp(s - lse[:, None])
        dp = do @ v[kj].T
        ds = p * (dp - dsum[:, None])
        dv = p.T @ do
        dk = scale * (ds.T @ q)
    return dq, dk, dv


def attend_bwd_given(q, k, v, do, o, lse, scale, q_rows=None, k_rows=None):
    """The same gradient formulas with O and LSE supplied by the caller.

    The backward of a CP shard runs on the final (merged) O and LSE of its
    rows, which another step produced and stored (the backward reading of the
    design notes); this entry takes them as inputs instead of recomputing
    them, so a stored (rounded) O or LSE enters exactly where it would:
      D_i   = dO_i . O_i                (O as given)
      P_ij  = exp(S_ij - LSE_i)         (LSE as given)
      dV_j  = sum_i P_ij dO_i
      dP_ij = dO_i . v_j
      dS_ij = P_ij (dP_ij - D_i)
      dQ_i  = scale * sum_j dS_ij k_j
      dK_j  = scale * sum_i dS_ij q_i
    q [Lq, d], k, v [Lk, d], do, o [Lq, d], lse [Lq].  With the exact O and
    LSE of ``attend`` this is ``attend_bwd``.  ``q_rows`` / ``k_rows`` select
    the returned rows as in ``attend_bwd``.
    """
    q, k, v, do, o, lse = _f64(q), _f64(k), _f64(v), _f64(do), _f64(o), _f64(lse)
    lq, lk = q.shape[0], k.shape[0]
    qi = np.arange(lq) if q_rows is None else np.asarray(q_rows, np.int64)
    kj = np.arange(lk) if k_rows is None else np.asarray(k_rows, np.int64)
    dq = np.zeros((qi.size, k.shape[1]), np.float64)
    dk = np.zeros((kj.size, q.shape[1]), np.float64)
    dv = np.zeros((kj.size, do.shape[1]), np.float64)
    if lq == 0 or lk == 0:
        return dq, dk, dv
    dsum = (do * o).sum(axis=1)
    if qi.size:
        s = scale * (q[qi] @ k.T)
        p = np.exp(s - lse[qi, None])
        ds = p * (do[qi] @ v.T - dsum[qi, None])
        dq = scale * (ds @ k)
    if kj.size:
        s = scale * (q @ k[kj].T)
        p = np.exp(s - lse[:, None])
        ds = p * (do @ v[kj].T - dsum[:, None])
        dv = p.T @ do
        dk = scale * (ds.T @ q)
    return dq, dk, dv


# ---------------------------------------------------------------------------
# Packed batches.  A descriptor is any mapping (or object) with the fields
#   cu_seqlens_q [nq+1], kind [nq] (0 whole, 1 shard), kv_first [nq],
#   kv_count [nq], cu_seqlens_k [nk+1], block_index [nk], num_slots
# (q_offset / k_offset are routing metadata and do not change any value).
# Packed tensors are THD: q [Tq, H, d], k and v [Tk, H, d].
# ---------------------------------------------------------------------------

def _field(desc, name):
    if isinstance(desc, dict):
        return desc[name]
    return getattr(desc, name)


def segment_rows(desc, s):
    """(first, last) packed query rows of segment s."""
    cq = _field(desc, "cu_seqlens_q")
    return int(cq[s]), int(cq[s + 1])


def _kv_rows(desc, j):
    ck = _field(desc, "cu_seqlens_k")
    return int(ck[j]), int(ck[j + 1])


def _segment_ranges(desc, s):
    first = int(_field(desc, "kv_first")[s])
    count = int(_field(desc, "kv_count")[s])
    return list(range(first, first + count))


def packed_forward(desc, q, k, v, scale, heads=None):
    """Forward of one coalesced launch over a packed whole+shard batch.

    Returns a dict of fp64 arrays; entries the launch does not write are NaN.
      out, lse        [Tq,H,d], [Tq,H]   whole rows: final output and LSE
      o_part, lse_part [S,Tq,H,d], [S,Tq,H]  shard rows: partial of the block
                       whose CP block index is the slot
      final_out, final_lse  every row's exact attention over all of its keys:
                       whole rows repeat out/lse; shard rows are computed
                       directly over the concatenation of the segment's
                       blocks (not through the merge), which is what the
                       merged result must equal.
    ``heads`` restricts the work to a subset of heads (others stay NaN).
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    tq, h_all, d = q.shape
    nslots = int(_field(desc, "num_slots"))
    kinds = _field(desc, "kind")
    bidx = _field(desc, "block_index")
    heads = range(h_all) if heads is None else heads
    res = {
        "out": np.full((tq, h_all, v.shape[2]), np.nan),
        "lse": np.full((tq, h_all), np.nan),
        "o_part": np.full((nslots, tq, h_all, v.shape[2]), np.nan),
        "lse_part": np.full((nslots, tq, h_all), np.nan),
        "final_out": np.full((tq, h_all, v.shape[2]), np.nan),
        "final_lse": np.full((tq, h_all), np.nan),
    }
    for s in range(len(kinds)):
        r0, r1 = segment_rows(desc, s)
        if r1 == r0:
            continue
        ranges = _segment_ranges(desc, s)
        for h in heads:
            qs = q[r0:r1, h]
            if int(kinds[s]) == WHOLE:
                k0, k1 = _kv_rows(desc, ranges[0])
                o, lse = attend(qs, k[k0:k1, h], v[k0:k1, h], scale)
                res["out"][r0:r1, h] = o
                res["lse"][r0:r1, h] = lse
                res["final_out"][r0:r1, h] = o
                res["final_lse"][r0:r1, h] = lse
            else:
                for j in ranges:
                    k0, k1 = _kv_rows(desc, j)
                    o, lse = attend(qs, k[k0:k1, h], v[k0:k1, h], scale)
                    b = int(bidx[j])
                    res["o_part"][b, r0:r1, h] = o
                    res["lse_part"][b, r0:r1, h] = lse
                kk = np.concatenate([k[slice(*_kv_rows(desc, j)), h] for j in ranges])
                vv = np.concatenate([v[slice(*_kv_rows(desc, j)), h] for j in ranges])
                o, lse = attend(qs, kk, vv, scale)
                res["final_out"][r0:r1, h] = o
                res["final_lse"][r0:r1, h] = lse
    return res


def packed_backward(desc, q, k, v, do, scale, heads=None):
    """Backward of the packed batch with respect to q, k, v.

    Each segment's loss term is sum(dO * O) over its rows, with O the final
    output (for a shard: attention over the concatenation of its blocks).
    Returns fp64 (dq [Tq,H,d], dk [Tk,H,d], dv [Tk,H,d]); rows no segment
    touches are zero.  A key range referenced by several segments receives
    the sum of their contributions.
    """
    q, k, v, do = _f64(q), _f64(k), _f64(v), _f64(do)
    tq, h_all, d = q.shape
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    heads = range(h_all) if heads is None else heads
    kinds = _field(desc, "kind")
    for s in range(len(kinds)):
        r0, r1 = segment_rows(desc, s)
        if r1 == r0:
            continue
        ranges = _segment_ranges(desc, s)
        bounds = [_kv_rows(desc, j) for j in ranges]
        for h in heads:
            kk = np.concatenate([k[a:b, h] for a, b in bounds])
            vv = np.concatenate([v[a:b, h] for a, b in bounds])
            g_q, g_k, g_v = attend_bwd(q[r0:r1, h], kk, vv, do[r0:r1, h], scale)
            dq[r0:r1, h] += g_q
            off = 0
            for a, b in bounds:
                dk[a:b, h] += g_k[off:off + (b - a)]
                dv[a:b, h] += g_v[off:off + (b - a)]
                off += b - a
    return dq, dk, dv
