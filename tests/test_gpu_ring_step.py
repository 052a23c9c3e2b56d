"""GPU parity of the ring-step forward (zl_attn_fwd_step): a shard sees one
K/V block per call and the epilogue folds it into a running fp32 (O, LSE)
(Sec. II-B, ring attention), with WHOLE fillers riding along in any step.
After the last step every shard row must equal exact attention over the
concatenation of its blocks, and every filler its own exact attention, to
the same tolerances as the all-blocks path (bf16: max|dO| <= 2e-2,
max|dLSE| <= 1e-3; fp32 plumbing: 1e-5)."""
import numpy as np
import pytest
import torch

import oracle
from tests._gpu import HAVE_GPU, api, to64

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="needs a GPU")]

O_TOL, LSE_TOL = 2e-2, 1e-3


def _ring(shard_q, shard_blocks, fillers, fill_step, H, hd, dtype, seed, block_index_fill=0):
    """shard_q: query count per shard; shard_blocks[s]: key counts of its blocks
    (all shards have the same number of blocks R); fillers: WHOLE lengths;
    fill_step[f]: the step that carries filler f; block_index_fill: the value
    of every block_index entry (a ring step does not read them)."""
    R = len(shard_blocks[0])
    g = torch.Generator().manual_seed(seed)
    rnd = lambda n: torch.randn((n, H, hd), generator=g).to(dtype)
    qs = [rnd(n) for n in shard_q]
    ks = [[rnd(n) for n in bl] for bl in shard_blocks]
    vs = [[rnd(n) for n in bl] for bl in shard_blocks]
    fq = [rnd(n) for n in fillers]
    fk = [rnd(n) for n in fillers]
    fv = [rnd(n) for n in fillers]
    scale = 1.0 / hd ** 0.5
    n_sq = sum(shard_q)
    max_tq = n_sq + max([sum(n for f, n in enumerate(fillers) if fill_step[f] == r) for r in range(R)] + [0])
    dev = "cuda"
    # a single step (FIRST|LAST) needs no accumulator: pass none
    o_acc = torch.full((max_tq, H, hd), float("nan"), device=dev) if R > 1 else None
    lse_acc = torch.full((max_tq, H), float("nan"), device=dev) if R > 1 else None
    shard_out = shard_lse = None
    fill_out = {}
    for r in range(R):
        fs = [f for f in range(len(fillers)) if fill_step[f] == r]
        lq = list(shard_q) + [fillers[f] for f in fs]
        lk = [bl[r] for bl in shard_blocks] + [fillers[f] for f in fs]
        kinds = [1] * len(shard_q) + [0] * len(fs)
        cu_q = np.concatenate([[0], np.cumsum(lq)]).astype(np.int32)
        cu_k = np.concatenate([[0], np.cumsum(lk)]).astype(np.int32)
        nseg = len(lq)
        desc = api.SegDesc(cu_q, np.array(kinds, np.uint8), np.arange(nseg, dtype=np.int32),
                           np.ones(nseg, np.int32), cu_k, np.full(nseg, block_index_fill, np.int32), 1)
        q = torch.cat(qs + [fq[f] for f in fs]).to(dev)
        k = torch.cat([ks[s][r] for s in range(len(shard_q))] + [fk[f] for f in fs]).to(dev)
        v = torch.cat([vs[s][r] for s in range(len(shard_q))] + [fv[f] for f in fs]).to(dev)
        out = torch.full_like(q, float("nan"))
        lse = torch.full((q.shape[0], H), float("nan"), device=dev)
        flags = (api.ZL_STEP_FIRST if r == 0 else 0) | (api.ZL_STEP_LAST if r == R - 1 else 0)
        api.attn_fwd_step(desc, q, k, v, scale, out, lse, o_acc, lse_acc, flags)
        torch.cuda.synchronize()
        row = n_sq
        for f in fs:
            fill_out[f] = (out[row:row + fillers[f]].clone(), lse[row:row + fillers[f]].clone())
            row += fillers[f]
        if r == R - 1:
            shard_out, shard_lse = out[:n_sq].clone(), lse[:n_sq].clone()
        # rows outside the shards are never touched in the accumulator
        if o_acc is not None:
            assert torch.isnan(o_acc[n_sq:]).all() and torch.isnan(lse_acc[n_sq:]).all()
    tol_o, tol_l = (1e-5, 1e-5) if dtype == torch.float32 else (O_TOL, LSE_TOL)
    row = 0
    for s, n in enumerate(shard_q):
        kk = torch.cat(ks[s]).double().numpy()
        vv = torch.cat(vs[s]).double().numpy()
        for h in range(H):
            o_ref, l_ref = oracle.attend(qs[s][:, h].double().numpy(), kk[:, h], vv[:, h], scale)
            np.testing.assert_allclose(to64(shard_out[row:row + n, h]), o_ref, rtol=0, atol=tol_o)
            np.testing.assert_allclose(to64(shard_lse[row:row + n, h]), l_ref, rtol=0, atol=tol_l)
        row += n
    for f, n in enumerate(fillers):
        o_got, l_got = fill_out[f]
        for h in range(H):
            o_ref, l_ref = oracle.attend(fq[f][:, h].double().numpy(), fk[f][:, h].double().numpy(),
                                         fv[f][:, h].double().numpy(), scale)
            np.testing.assert_allclose(to64(o_got[:, h]), o_ref, rtol=0, atol=tol_o)
            np.testing.assert_allclose(to64(l_got[:, h]), l_ref, rtol=0, atol=tol_l)


@pytest.mark.parametrize("hd", [64, 128])
def test_ring_steps_bf16(hd):
    # two shards over four blocks each (one block empty, ragged sizes), fillers in steps 0, 1, 3
    _ring(shard_q=(150, 33), shard_blocks=((300, 0, 129, 64), (64, 191, 1, 256)), fillers=(200, 77, 1),
          fill_step=(0, 1, 3), H=2, hd=hd, dtype=torch.bfloat16, seed=31)


def test_ring_steps_ignore_block_index():
    """A ring step reads no block_index: with every entry -1 (a sentinel a caller might leave there) the
    shard rows still fold into the accumulator and match the oracle.  (The step plan once took the shard
    items' slot from block_index, and a negative slot sent them down the WHOLE epilogue.)"""
    _ring(shard_q=(150, 33), shard_blocks=((300, 0, 129), (64, 191, 1)), fillers=(200,), fill_step=(1,), H=2,
          hd=128, dtype=torch.bfloat16, seed=36, block_index_fill=-1)


def test_ring_steps_first_block_empty_bf16():
    _ring(shard_q=(97,), shard_blocks=((0, 130, 0),), fillers=(), fill_step=(), H=3, hd=128,
          dtype=torch.bfloat16, seed=32)


def test_ring_single_step_bf16():
    # FIRST|LAST in one call: no accumulator needed at all
    _ring(shard_q=(129,), shard_blocks=((257,),), fillers=(64,), fill_step=(0,), H=2, hd=128,
          dtype=torch.bfloat16, seed=33)


def test_ring_steps_fp32():
    _ring(shard_q=(70, 5), shard_blocks=((64, 33, 0), (128, 1, 7)), fillers=(40,), fill_step=(2,), H=2, hd=64,
          dtype=torch.float32, seed=34)


def test_all_gather_mode_matches_all_blocks_mode():
    """All-gather mode (Tab. II (q,1,1)): each shard attends once to the concatenation of its blocks
    (one range, zl_attn_fwd_step with FIRST|LAST): no partials, no merge.  It must agree with the
    all-blocks launch plus LSE merge on the same inputs, and with the oracle."""
    from tests import _descs
    d = _descs.mixed_small()          # shard 3 has blocks of 300, 0 and 129 keys, consecutive in K
    H, hd = 2, 128
    g = torch.Generator().manual_seed(35)
    tq, tk = d["cu_seqlens_q"][-1], d["cu_seqlens_k"][-1]
    q, k, v = (torch.randn((n, H, hd), generator=g).to(torch.bfloat16) for n in (tq, tk, tk))
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    scale = 1.0 / hd ** 0.5
    desc = api.SegDesc.of(d)
    out_b, lse_b, op, lp = api.attn_fwd(desc, qd, kd, vd, scale)
    api.lse_merge(desc, op, lp, out_b, lse_b)
    # gathered descriptor: every segment keeps its consecutive ranges as one
    cu_k, first = [0], []
    for s in range(len(d["kind"])):
        j0, j1 = d["kv_first"][s], d["kv_first"][s] + d["kv_count"][s]
        first.append(len(cu_k) - 1)
        cu_k.append(cu_k[-1] + d["cu_seqlens_k"][j1] - d["cu_seqlens_k"][j0])
    n = len(d["kind"])
    gdesc = api.SegDesc(np.asarray(d["cu_seqlens_q"], np.int32), np.asarray(d["kind"], np.uint8),
                        np.asarray(first, np.int32), np.ones(n, np.int32), np.asarray(cu_k, np.int32),
                        np.zeros(n, np.int32), 1)
    out_g = torch.full_like(qd, float("nan"))
    lse_g = torch.full((tq, H), float("nan"), device="cuda")
    api.attn_fwd_step(gdesc, qd, kd, vd, scale, out_g, lse_g, None, None, api.ZL_STEP_FIRST | api.ZL_STEP_LAST)
    torch.cuda.synchronize()
    rows = np.arange(tq)
    np.testing.assert_allclose(to64(out_g[rows]), to64(out_b[rows]), rtol=0, atol=O_TOL)
    np.testing.assert_allclose(to64(lse_g[rows]), to64(lse_b[rows]), rtol=0, atol=LSE_TOL)
    ref = oracle.packed_forward(d, q.double().numpy(), k.double().numpy(), v.double().numpy(), scale)
    np.testing.assert_allclose(to64(out_g), ref["final_out"], rtol=0, atol=O_TOL)
    np.testing.assert_allclose(to64(lse_g), ref["final_lse"], rtol=0, atol=LSE_TOL)


def _bwd_tol_check(got, ref, name):
    got, ref = to64(got), np.asarray(ref)
    err = np.abs(got - ref).max()
    assert err <= 2e-2 * max(1.0, np.abs(ref).max()), f"{name}: max abs err {err}"
    nref = np.linalg.norm(ref)
    assert nref == 0 or np.linalg.norm(got - ref) / nref <= 1e-2, name   # the all-blocks path's bound


@pytest.mark.parametrize("hd,fill_step", [(128, 0), (64, 2), (128, 1)])
def test_ring_backward_steps_match_all_blocks_backward(hd, fill_step):
    """zl_attn_bwd_step over a shard's blocks, one per call (FIRST ... LAST),
    with the WHOLE fillers riding in one step.  Every block's dK/dV and the
    fillers' dQ/dK/dV are the same work items as in the all-blocks backward
    and must match it bit for bit; the shard's dQ is summed block by block in
    fp32 and must match the all-blocks dQ and the oracle to the backward
    tolerances."""
    H = 2
    blocks = (129, 64, 200)          # the shard's K/V blocks, consecutive in K
    nq, fills = 150, (77, 64, 1)
    g = torch.Generator().manual_seed(40 + hd + fill_step)
    R = len(blocks)
    tq, tk = nq + sum(fills), sum(blocks) + sum(fills)
    q, do = (torch.randn((tq, H, hd), generator=g).to(torch.bfloat16) for _ in range(2))
    k, v = (torch.randn((tk, H, hd), generator=g).to(torch.bfloat16) for _ in range(2))
    scale = 1.0 / hd ** 0.5
    # all-blocks layout: the shard (rows 0..nq, ranges 0..R-1), then the fillers
    lq = [nq] + list(fills)
    cu_q = np.concatenate([[0], np.cumsum(lq)]).astype(np.int32)
    cu_k = np.concatenate([[0], np.cumsum(list(blocks) + list(fills))]).astype(np.int32)
    d = dict(cu_seqlens_q=tuple(cu_q), kind=(1,) + (0,) * len(fills),
             kv_first=(0,) + tuple(R + i for i in range(len(fills))), kv_count=(R,) + (1,) * len(fills),
             cu_seqlens_k=tuple(cu_k), block_index=tuple(range(R)) + (0,) * len(fills), num_slots=R,
             q_offset=None, k_offset=None)
    desc = api.SegDesc.of(d)
    qd, kd, vd, dod = q.cuda(), k.cuda(), v.cuda(), do.cuda()
    out, lse, op, lp = api.attn_fwd(desc, qd, kd, vd, scale)
    api.lse_merge(desc, op, lp, out, lse)
    dq_ref, dk_ref, dv_ref = api.attn_bwd(desc, qd, kd, vd, out, lse, dod, scale)

    dq = torch.full_like(qd, float("nan"))
    dq_acc = torch.full((tq, H, hd), float("nan"), device="cuda")
    nf = len(fills)
    for r in range(R):
        with_fill = r == fill_step
        rows = tq if with_fill else nq
        b0, b1 = int(cu_k[r]), int(cu_k[r + 1])
        ks = [kd[b0:b1]] + ([kd[cu_k[R]:]] if with_fill else [])
        vs = [vd[b0:b1]] + ([vd[cu_k[R]:]] if with_fill else [])
        kr, vr = torch.cat(ks), torch.cat(vs)
        lk = [b1 - b0] + (list(fills) if with_fill else [])
        nseg = 1 + (nf if with_fill else 0)
        sdesc = api.SegDesc(cu_q[:nseg + 1].copy(), np.array([1] + [0] * (nseg - 1), np.uint8),
                            np.arange(nseg, dtype=np.int32), np.ones(nseg, np.int32),
                            np.concatenate([[0], np.cumsum(lk)]).astype(np.int32), np.zeros(nseg, np.int32), 1)
        dkr = torch.full_like(kr, float("nan"))
        dvr = torch.full_like(vr, float("nan"))
        flags = (api.ZL_STEP_FIRST if r == 0 else 0) | (api.ZL_STEP_LAST if r == R - 1 else 0)
        api.attn_bwd_step(sdesc, qd[:rows], kr, vr, out[:rows], lse[:rows], dod[:rows], scale, dq[:rows], dkr, dvr,
                          dq_acc, flags)
        torch.cuda.synchronize()
        assert torch.equal(dkr[:b1 - b0], dk_ref[b0:b1]) and torch.equal(dvr[:b1 - b0], dv_ref[b0:b1]), r
        if with_fill:
            assert torch.equal(dkr[b1 - b0:], dk_ref[cu_k[R]:]) and torch.equal(dvr[b1 - b0:], dv_ref[cu_k[R]:])
            assert torch.equal(dq[nq:], dq_ref[nq:])
    _bwd_tol_check(dq[:nq], to64(dq_ref[:nq]), "ring dq vs all-blocks dq")
    rq, _, _ = oracle.packed_backward(d, q.double().numpy(), k.double().numpy(), v.double().numpy(),
                                      do.double().numpy(), scale)
    _bwd_tol_check(dq, rq, "ring dq vs oracle")


def test_single_backward_step_equals_backward():
    """flags = FIRST|LAST (no accumulator) is the ordinary backward, bit for bit."""
    H, hd = 2, 128
    d = dict(cu_seqlens_q=(0, 97, 161), kind=(1, 0), kv_first=(0, 1), kv_count=(1, 1),
             cu_seqlens_k=(0, 257, 321), block_index=(0, 0), num_slots=1, q_offset=None, k_offset=None)
    g = torch.Generator().manual_seed(44)
    q, do = (torch.randn((161, H, hd), generator=g).to(torch.bfloat16).cuda() for _ in range(2))
    k, v = (torch.randn((321, H, hd), generator=g).to(torch.bfloat16).cuda() for _ in range(2))
    desc = api.SegDesc.of(d)
    scale = hd ** -0.5
    out, lse, op, lp = api.attn_fwd(desc, q, k, v, scale)
    api.lse_merge(desc, op, lp, out, lse)
    dq_ref, dk_ref, dv_ref = api.attn_bwd(desc, q, k, v, out, lse, do, scale)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    api.attn_bwd_step(desc, q, k, v, out, lse, do, scale, dq, dk, dv, None, api.ZL_STEP_FIRST | api.ZL_STEP_LAST)
    torch.cuda.synchronize()
    assert torch.equal(dq, dq_ref) and torch.equal(dk, dk_ref) and torch.equal(dv, dv_ref)


@pytest.mark.parametrize("seed", range(4))
def test_ring_steps_random_bf16(seed):
    """Random ring shapes: 1-2 shards of up to 700 queries, 2-5 blocks of up
    to 700 keys (some empty), 0-4 fillers in random steps, both head dims."""
    rng = np.random.default_rng(700 + seed)
    R = int(rng.integers(2, 6))
    nsh = int(rng.integers(1, 3))
    shard_q = tuple(int(rng.integers(1, 701)) for _ in range(nsh))
    shard_blocks = tuple(tuple(int(rng.integers(0, 701)) for _ in range(R)) for _ in range(nsh))
    nf = int(rng.integers(0, 5))
    fillers = tuple(int(rng.integers(1, 701)) for _ in range(nf))
    fill_step = tuple(int(rng.integers(0, R)) for _ in range(nf))
    _ring(shard_q, shard_blocks, fillers, fill_step, H=2, hd=(64, 128)[seed % 2], dtype=torch.bfloat16,
          seed=800 + seed)
