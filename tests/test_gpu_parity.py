"""GPU parity: the HIP path against the fp64 oracle, element by element, on
small seeded batches that span several tiles and ragged tails, plus the
invariants exact attention must satisfy on the device itself.

Tolerances: bf16 max|dO| <= 2e-2 and max|dLSE| <= 1e-3 for outputs; backward
max abs error <= 2e-2 * max(1, max|ref|) and relative Frobenius error <= 1e-2
(see BWD_REL_FRO); fp32 plumbing runs 1e-5 on both.
"""
import numpy as np
import pytest
import torch

import oracle
from tests import _descs
from tests._gpu import HAVE_GPU, api, to64

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="needs a GPU")]

O_TOL, LSE_TOL = 2e-2, 1e-3
# Backward, end to end through the bf16 forward, on whole small batches: the
# CPU error budget (tests/test_bwd_error_budget.py) puts the chain at 0.24% on
# unscaled inputs and about 0.6% on x4-scaled ones (a nearly one-hot softmax,
# where dS = P (dP - D) is a small difference and the bf16-stored O's error
# through D counts most), so the relative Frobenius bound is 1e-2.
BWD_REL_FRO = 1e-2


def _inputs(d, H, hd, dtype, seed):
    g = torch.Generator().manual_seed(seed)
    tq, tk = d["cu_seqlens_q"][-1], d["cu_seqlens_k"][-1]
    q, k, v, do = (torch.randn((n, H, hd), generator=g).to(dtype) for n in (tq, tk, tk, tq))
    return q, k, v, do


def _check_bwd(got, ref, name):
    got, ref = to64(got), np.asarray(ref)
    err = np.abs(got - ref).max() if ref.size else 0.0
    bound = 2e-2 * max(1.0, np.abs(ref).max() if ref.size else 0.0)
    assert err <= bound, f"{name}: max abs err {err} > {bound}"
    nref = np.linalg.norm(ref)
    if nref > 0:
        rel = np.linalg.norm(got - ref) / nref
        assert rel <= BWD_REL_FRO, f"{name}: relative Frobenius err {rel}"
        print(f"{name}: rel Frobenius {rel:.3g}", flush=True)


def _whole_rows(d):
    rows = []
    for s, kd in enumerate(d["kind"]):
        if kd == 0:
            rows += list(range(d["cu_seqlens_q"][s], d["cu_seqlens_q"][s + 1]))
    return np.array(rows, dtype=np.int64)


def _shard_rows_slots(d):
    out = []
    for s, kd in enumerate(d["kind"]):
        if kd == 1:
            r = np.arange(d["cu_seqlens_q"][s], d["cu_seqlens_q"][s + 1])
            slots = [d["block_index"][j] for j in range(d["kv_first"][s], d["kv_first"][s] + d["kv_count"][s])]
            out.append((r, slots))
    return out


def run_and_compare(d, H, hd, dtype, seed, backward=True, scale=None, part_dtype=torch.float32):
    desc = api.SegDesc.of(d)
    q, k, v, do = _inputs(d, H, hd, dtype, seed)
    scale = 1.0 / hd ** 0.5 if scale is None else scale
    qd, kd_, vd, dod = (t.cuda() for t in (q, k, v, do))
    tq = q.shape[0]
    nan = float("nan")
    out = torch.full_like(qd, nan)
    lse = torch.full((tq, H), nan, device="cuda")
    o_part = torch.full((max(desc.num_slots, 1), tq, H, hd), nan, dtype=part_dtype, device="cuda")
    lse_part = torch.full((max(desc.num_slots, 1), tq, H), nan, device="cuda")
    api.attn_fwd(desc, qd, kd_, vd, scale, out, lse, o_part if desc.num_slots else None,
                 lse_part if desc.num_slots else None)
    torch.cuda.synchronize()
    ref = oracle.packed_forward(d, q.double().numpy(), k.double().numpy(), v.double().numpy(), scale)
    tol_o, tol_l = (1e-5, 1e-5) if dtype == torch.float32 else (O_TOL, LSE_TOL)

    wr = _whole_rows(d)
    if wr.size:
        np.testing.assert_allclose(to64(out)[wr], ref["out"][wr], rtol=0, atol=tol_o)
        np.testing.assert_allclose(to64(lse)[wr], ref["lse"][wr], rtol=0, atol=tol_l)
    for rows, slots in _shard_rows_slots(d):
        # shard rows are not written to out by the forward
        assert torch.isnan(out[torch.as_tensor(rows, device="cuda")]).all()
        for b in slots:
            got_l = to64(lse_part[b])[rows]
            ref_l = ref["lse_part"][b][rows]
            assert np.array_equal(np.isneginf(got_l), np.isneginf(ref_l))
            fin = np.isfinite(ref_l)
            np.testing.assert_allclose(got_l[fin], ref_l[fin], rtol=0, atol=tol_l)
            np.testing.assert_allclose(to64(o_part[b])[rows], ref["o_part"][b][rows], rtol=0, atol=tol_o)
    if wr.size and desc.num_slots:
        # whole rows are never written to the partials
        assert torch.isnan(o_part[:, torch.as_tensor(wr, device="cuda")]).all()

    if desc.num_slots:
        api.lse_merge(desc, o_part, lse_part, out, lse)
        torch.cuda.synchronize()
    fin = ~np.isnan(ref["final_out"][:, 0, 0])
    np.testing.assert_allclose(to64(out)[fin], ref["final_out"][fin], rtol=0, atol=tol_o)
    np.testing.assert_allclose(to64(lse)[fin], ref["final_lse"][fin], rtol=0, atol=tol_l)

    if backward:
        dq, dk, dv = api.attn_bwd(desc, qd, kd_, vd, out, lse, dod, scale)
        torch.cuda.synchronize()
        rq, rk, rv = oracle.packed_backward(d, q.double().numpy(), k.double().numpy(), v.double().numpy(),
                                            do.double().numpy(), scale)
        _check_bwd(dq, rq, "dq")
        _check_bwd(dk, rk, "dk")
        _check_bwd(dv, rv, "dv")
    return out, lse


@pytest.mark.parametrize("hd", [64, 128])
def test_bf16_partials(hd):
    """Partials stored in bf16 (zl_attn_fwd_ex / zl_lse_merge_ex): each O_b is rounded once more, the
    same bf16 tolerances against the oracle hold, and the merged output stays within that tolerance of the
    fp32-partial path's (an absolute bound: blocks may cancel, so |O| can be far below |O_b|)."""
    d = _descs.mixed_small()
    out_b, lse_b = run_and_compare(d, 3, hd, torch.bfloat16, 41 + hd, backward=False, part_dtype=torch.bfloat16)
    out_f, lse_f = run_and_compare(d, 3, hd, torch.bfloat16, 41 + hd, backward=False)
    assert torch.equal(lse_b, lse_f)  # the LSE partials stay fp32
    assert (out_b.float() - out_f.float()).abs().max().item() <= O_TOL


@pytest.mark.parametrize("seed", range(3))
def test_bf16_partials_random_descriptors(seed):
    rng = np.random.default_rng(700 + seed)
    d = _descs.random_desc(rng, int(rng.integers(0, 3)), int(rng.integers(1, 4)), 300, 5)
    run_and_compare(d, 2, 128, torch.bfloat16, 90 + seed, backward=True, part_dtype=torch.bfloat16)


def test_mfma_layout_probe_free_smoke():
    """One whole segment of exactly one tile: the simplest possible launch."""
    d = _descs.desc((0, 128), (0,), (0,), (1,), (0, 128), (0,), 0)
    run_and_compare(d, 1, 128, torch.bfloat16, 1)


@pytest.mark.parametrize("hd", [64, 128])
def test_mixed_small_bf16(hd):
    run_and_compare(_descs.mixed_small(), 3, hd, torch.bfloat16, 11 + hd)


@pytest.mark.parametrize("hd", [64, 128])
def test_mixed_small_fp32_forward(hd):
    run_and_compare(_descs.mixed_small(), 2, hd, torch.float32, 5 + hd, backward=False)


def test_tiny_plumbing_fp32():
    """The fp32 plumbing workload: whole 64/128/256 and four 64-query shards
    sharing four 64-key blocks, merged."""
    from paper_2608_01150_amd import workloads as W
    w = W.get("c1")
    d = w.desc_dict()
    desc = api.SegDesc.of(w)
    q, k, v = (w.full(t) for t in (W.TENSOR_Q, W.TENSOR_K, W.TENSOR_V))
    out, lse, o_part, lse_part = api.attn_fwd(desc, q.cuda(), k.cuda(), v.cuda(), w.scale)
    api.lse_merge(desc, o_part, lse_part, out, lse)
    torch.cuda.synchronize()
    ref = oracle.packed_forward(d, q.double().numpy(), k.double().numpy(), v.double().numpy(), w.scale)
    np.testing.assert_allclose(to64(out), ref["final_out"], rtol=0, atol=1e-5)
    np.testing.assert_allclose(to64(lse), ref["final_lse"], rtol=0, atol=1e-5)
    for b in range(4):
        np.testing.assert_allclose(to64(o_part[b])[448:], ref["o_part"][b][448:], rtol=0, atol=1e-5)


@pytest.mark.parametrize("seed", range(4))
def test_random_descriptors_bf16(seed):
    rng = np.random.default_rng(100 + seed)
    d = _descs.random_desc(rng, 3, 2, 400, 4)
    if not d["kind"] or d["cu_seqlens_q"][-1] == 0:
        pytest.skip("empty draw")
    run_and_compare(d, 2, 128 if seed % 2 else 64, torch.bfloat16, seed)


def test_edge_lengths_bf16():
    """1-row segment, 1-key block, lengths around the 32/64/128 tile edges."""
    d = _descs.desc(cu_q=(0, 1, 64, 193, 320, 385), kind=(0, 0, 0, 1, 1),
                    kv_first=(0, 1, 2, 3, 5), kv_count=(1, 1, 1, 2, 2),
                    cu_k=(0, 1, 64, 193, 194, 257, 322, 450), block_index=(0, 0, 0, 1, 0, 0, 1), num_slots=2)
    run_and_compare(d, 2, 128, torch.bfloat16, 3)


def test_tiny_softmax_scale_masks_exactly():
    """Any finite positive scale is valid; at 1e-30 every score is ~0, so keys
    past a range must be masked by -inf itself (a large finite negative score
    would shrink to O(1) after scaling and take softmax weight)."""
    d = _descs.desc(cu_q=(0, 1, 64, 193, 320, 385), kind=(0, 0, 0, 1, 1),
                    kv_first=(0, 1, 2, 3, 5), kv_count=(1, 1, 1, 2, 2),
                    cu_k=(0, 1, 64, 193, 194, 257, 322, 450), block_index=(0, 0, 0, 1, 0, 0, 1), num_slots=2)
    run_and_compare(d, 2, 128, torch.bfloat16, 5, scale=1e-30)


def test_constant_v_returns_that_row():
    d = _descs.mixed_small()
    desc = api.SegDesc.of(d)
    H, hd = 2, 128
    q, k, _, _ = _inputs(d, H, hd, torch.bfloat16, 9)
    row = torch.randn(H, hd, generator=torch.Generator().manual_seed(3)).to(torch.bfloat16)
    v = row.expand(k.shape[0], H, hd).contiguous()
    out, lse, o_part, lse_part = api.attn_fwd(desc, q.cuda(), k.cuda(), v.cuda(), 0.1)
    api.lse_merge(desc, o_part, lse_part, out, lse)
    torch.cuda.synchronize()
    expect = row.float().cuda().expand_as(out)
    assert (out.float() - expect).abs().max().item() <= 1e-2


def test_segment_isolation_and_determinism():
    """Perturbing one segment leaves every other segment's outputs bit-identical
    (Sec. IV-D keeps sequences separate); repeated runs are bit-identical."""
    d = _descs.mixed_small()
    desc = api.SegDesc.of(d)
    H, hd = 2, 128
    q, k, v, _ = _inputs(d, H, hd, torch.bfloat16, 21)
    a = api.attn_fwd(desc, q.cuda(), k.cuda(), v.cuda(), 0.1)
    b = api.attn_fwd(desc, q.cuda(), k.cuda(), v.cuda(), 0.1)
    torch.cuda.synchronize()
    # written regions only: whole rows of out/lse, slots 2,0,1 of rows 277..427, slot 0 of rows 427..460
    def written(r):
        return (r[0][:277], r[1][:277], r[2][[2, 0, 1], 277:427], r[3][[2, 0, 1], 277:427],
                r[2][0, 427:460], r[3][0, 427:460])
    for x, y in zip(written(a), written(b)):
        assert torch.equal(x, y)
    q2, k2, v2 = q.clone(), k.clone(), v.clone()
    q2[200:277] *= -1
    k2[200:277] += 1
    v2[200:277] -= 2
    c = api.attn_fwd(desc, q2.cuda(), k2.cuda(), v2.cuda(), 0.1)
    torch.cuda.synchronize()
    wa, wc = written(a), written(c)
    assert torch.equal(wa[0][:200], wc[0][:200]) and torch.equal(wa[1][:200], wc[1][:200])
    for x, y in zip(wa[2:], wc[2:]):
        assert torch.equal(x, y)
    assert not torch.equal(a[0][200:277], c[0][200:277])


def test_ring_step_mode_equals_all_blocks_mode():
    """A shard against all of its blocks in one launch gives the same partials,
    bit for bit, as one launch per block (the ring's per-step call)."""
    d = _descs.desc(cu_q=(0, 300), kind=(1,), kv_first=(0,), kv_count=(3,),
                    cu_k=(0, 200, 456, 500), block_index=(2, 0, 1), num_slots=3)
    H, hd = 2, 128
    q, k, v, _ = _inputs(d, H, hd, torch.bfloat16, 4)
    qd, kd_, vd = q.cuda(), k.cuda(), v.cuda()
    _, _, o_all, l_all = api.attn_fwd(api.SegDesc.of(d), qd, kd_, vd, 0.09)
    o_step = torch.empty_like(o_all)
    l_step = torch.empty_like(l_all)
    for j, b in enumerate((2, 0, 1)):
        dj = _descs.desc(cu_q=(0, 300), kind=(1,), kv_first=(j,), kv_count=(1,),
                         cu_k=(0, 200, 456, 500), block_index=(2, 0, 1), num_slots=3)
        api.attn_fwd(api.SegDesc.of(dj), qd, kd_, vd, 0.09, None, None, o_step, l_step)
    torch.cuda.synchronize()
    assert torch.equal(o_all, o_step) and torch.equal(l_all, l_step)


@pytest.mark.parametrize("seed", range(6))
def test_random_descriptors_larger_bf16(seed):
    """Larger random packed batches (up to 1100 rows per segment or block,
    several tiles and ragged tails everywhere), both head dims, more heads."""
    rng = np.random.default_rng(500 + seed)
    d = _descs.random_desc(rng, 4, 2, 1100, 5)
    if not d["kind"] or d["cu_seqlens_q"][-1] == 0:
        pytest.skip("empty draw")
    run_and_compare(d, 3, (64, 128)[seed % 2], torch.bfloat16, 600 + seed)


def test_backward_zero_row_shard_writes_zero_dkdv():
    """The blocks of a SHARD segment without query rows get dK = dV = 0 (no query attends to them),
    written by the backward: the buffers start as NaN.  The WHOLE segments around it match the oracle."""
    d = _descs.desc(cu_q=(0, 150, 150, 190), kind=(0, 1, 0), kv_first=(0, 1, 3), kv_count=(1, 2, 1),
                    cu_k=(0, 150, 350, 420, 460), block_index=(0, 0, 1, 0), num_slots=2)
    H, hd = 2, 128
    desc = api.SegDesc.of(d)
    q, k, v, do = _inputs(d, H, hd, torch.bfloat16, 61)
    qd, kd_, vd, dod = (t.cuda() for t in (q, k, v, do))
    scale = hd ** -0.5
    out, lse, _, _ = api.attn_fwd(desc, qd, kd_, vd, scale)
    nan = float("nan")
    dq = torch.full_like(qd, nan)
    dk, dv = torch.full_like(kd_, nan), torch.full_like(vd, nan)
    api.attn_bwd(desc, qd, kd_, vd, out, lse, dod, scale, dq, dk, dv)
    torch.cuda.synchronize()
    assert torch.count_nonzero(dk[150:420]) == 0 and torch.count_nonzero(dv[150:420]) == 0
    rq, rk, rv = oracle.packed_backward(d, q.double().numpy(), k.double().numpy(), v.double().numpy(),
                                        do.double().numpy(), scale)
    assert not np.isnan(to64(dq)).any()
    _check_bwd(dq, rq, "dq")
    _check_bwd(dk, rk, "dk")
    _check_bwd(dv, rv, "dv")


def test_backward_without_query_rows():
    """Tq = 0: the only segment is a SHARD with no queries over two blocks; the call launches no
    preprocess (nothing to reduce) and still zeroes both blocks' dK/dV."""
    d = _descs.desc(cu_q=(0, 0), kind=(1,), kv_first=(0,), kv_count=(2,), cu_k=(0, 64, 100),
                    block_index=(0, 1), num_slots=2)
    H, hd = 3, 64
    desc = api.SegDesc.of(d)
    g = torch.Generator().manual_seed(62)
    k, v = (torch.randn((100, H, hd), generator=g).to(torch.bfloat16).cuda() for _ in range(2))
    empty = torch.empty((0, H, hd), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((0, H), dtype=torch.float32, device="cuda")
    dk, dv = torch.full_like(k, float("nan")), torch.full_like(v, float("nan"))
    api.attn_bwd(desc, empty, k, v, empty, lse, empty, hd ** -0.5, empty, dk, dv)
    torch.cuda.synchronize()
    assert torch.count_nonzero(dk) == 0 and torch.count_nonzero(dv) == 0


def test_forward_running_max_jumps():
    """The forward exponentiates a block against the running maximum as it stands and rescales only when
    the block's sum of exponentials passes 2^64.  All queries share one direction u; keys that are
    multiples f*u score about 17.8*f (log2 units) against ~5 for the others.  In a 600-key segment the
    maximum then rises by ~13 (key 40, block 1 of tile 0: common path, P up to 2^13), ~89 (key 200,
    block 0 of tile 3: slow path), ~54 (key 300, block 1 of tile 4: common path with P near 2^54), ~89
    (key 500, block 1 of tile 7: slow path after block 0 has entered O) and ~107 (key 530, block 0 of
    tile 8: slow path).  An 80-key segment jumps by ~48 in its second tile (common path).  Both must
    match the oracle."""
    H, hd = 2, 128
    g = torch.Generator().manual_seed(63)
    u = torch.randn((1, H, hd), generator=g)
    d = _descs.desc(cu_q=(0, 600, 680), kind=(0, 0), kv_first=(0, 1), kv_count=(1, 1), cu_k=(0, 600, 680),
                    block_index=(0, 0), num_slots=0)
    q = (u + 0.05 * torch.randn((680, H, hd), generator=g)).to(torch.bfloat16)
    k = torch.randn((680, H, hd), generator=g)
    v = torch.randn((680, H, hd), generator=g).to(torch.bfloat16)
    for key, f in ((40, 1.0), (200, 6.0), (300, 9.0), (500, 14.0), (530, 20.0), (600 + 70, 3.0)):
        k[key] = f * u[0]
    k = k.to(torch.bfloat16)
    desc = api.SegDesc.of(d)
    scale = hd ** -0.5
    out, lse, _, _ = api.attn_fwd(desc, q.cuda(), k.cuda(), v.cuda(), scale)
    torch.cuda.synchronize()
    ref = oracle.packed_forward(d, q.double().numpy(), k.double().numpy(), v.double().numpy(), scale)
    np.testing.assert_allclose(to64(out), ref["out"], rtol=0, atol=O_TOL)
    np.testing.assert_allclose(to64(lse), ref["lse"], rtol=0, atol=LSE_TOL)
