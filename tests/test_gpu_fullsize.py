"""GPU parity at the benchmark's full sizes, in the launch configuration
bench.py times (one forward over the whole packed batch, the LSE merge, the
backward), checked on seeded samples the fp64 oracle computes one by one:

  * forward and dQ on 64 sampled query rows of sampled segments, on EVERY
    head: the first and last rows, both sides of the 64-, 128-, 256- and
    512-row tile edges (rows 63/64, 127/128, 255/256, 511/512) and seeded
    rows; a shard row is checked per block (partial O_b, LSE_b) and after the
    merge against attention over the concatenation of its blocks.  Output and
    LSE are checked per head; dQ's max abs error and relative Frobenius error
    over the sampled rows of all heads of a segment together (the scale
    max|ref| and the Frobenius ratio of a handful of rows of a nearly one-hot
    segment swing with the sample, see tests/test_bwd_error_budget.py);
  * on one seeded head, EVERY query row of the segment (output, LSE, per-block
    partials of a shard, dQ) and dK, dV on sampled keys, which need the
    oracle's O and LSE for every query of the segment anyway; for the
    31,110 x 497,760 shard this is too slow on the host, so there it is
    replaced by identities that hold at any size (sum over all keys of dK =
    0, sum over all keys of dV = sum over queries of dO) checked on every
    head.

Inputs come from the seeded counter-based generator, drawn on the GPU (by
torch, not by the library) for the launch.  The oracle reads those same
tensors back per head, after a seeded sample of their rows has been checked
bit for bit against the generator run on the CPU.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_01150_amd import workloads as W
from tests._gpu import HAVE_GPU, api, to64

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="needs a GPU")]

O_TOL, LSE_TOL = 2e-2, 1e-3
# Backward end to end (through the bf16 forward), relative Frobenius error of the small per-head samples
# (two dozen keys of dK/dV): 2e-2.  The CPU error budget (tests/test_bwd_error_budget.py) puts the chain at
# 0.24% on unscaled inputs and 0.5-0.6% on the x4-scaled video, but over a small sample of that video the
# ratio spreads around it (1.2% at p99.9 over 64 rows).
BWD_REL_FRO = 2e-2
# Over large samples (every row of a head, or a segment's sampled rows of all heads) the spread is small and
# the bound is 1e-2: the budget's end-to-end chain on the x4 video is 0.59%, and the GPU measures 0.57% there.
BWD_REL_FRO_POOLED = 1e-2

# segments checked per workload, and whether dK/dV of the shard is sampled
PLAN = {
    "c2": dict(segments=(0, 7, 15), shard_dkdv=True),
    "c3": dict(segments=None, shard_dkdv=True),       # None: the scaled segment, a 3600 and the last 1560
    "c4": dict(segments=(0, 1, 6), shard_dkdv=True),
    "c5": dict(segments=(0, 1, 12), shard_dkdv=False),
}
EDGES = (0, 1, 63, 64, 127, 128, 255, 256, 511, 512)


def _run(w):
    dev = torch.device("cuda:0")
    desc = api.SegDesc.of(w)
    q, k, v, do = (w.full(t, device=dev) for t in (W.TENSOR_Q, W.TENSOR_K, W.TENSOR_V, W.TENSOR_DO))
    out, lse, o_part, lse_part = api.attn_fwd(desc, q, k, v, w.scale)
    parts = None
    if w.num_slots:
        parts = (o_part, lse_part)
        api.lse_merge(desc, o_part, lse_part, out, lse)
    dq, dk, dv = api.attn_bwd(desc, q, k, v, out, lse, do, w.scale)
    torch.cuda.synchronize()
    return dict(q=q, k=k, v=v, do=do, out=out, lse=lse, parts=parts, dq=dq, dk=dk, dv=dv)


def _check_inputs_match_cpu_draw(w, res, rng):
    """The device-drawn inputs equal the CPU generator bit for bit on seeded rows (all heads)."""
    for t, name, n in ((W.TENSOR_Q, "q", w.total_q), (W.TENSOR_K, "k", w.total_k), (W.TENSOR_V, "v", w.total_k),
                       (W.TENSOR_DO, "do", w.total_q)):
        for r in sorted(set(rng.choice(n, size=8, replace=False).tolist()) | {0, n - 1}):
            assert torch.equal(res[name][r:r + 1].cpu(), w.slice(t, r, r + 1)), f"{name} row {r}"


def _ranges(w, s):
    return [(w.cu_seqlens_k[j], w.cu_seqlens_k[j + 1], w.block_index[j])
            for j in range(w.kv_first[s], w.kv_first[s] + w.kv_count[s])]


def _rows(rng, a, b, extra=54):
    n = b - a
    base = {min(n - 1, e) for e in EDGES} | {n - 1}
    base |= set(rng.choice(n, size=min(n, extra), replace=False).tolist())
    return np.array(sorted(base), dtype=np.int64)


def _host(t, rows_or_slice, h):
    """fp64 host copy of head h of a device tensor [T, H, d] at the given rows."""
    return t[rows_or_slice, h].double().cpu().numpy()


def _bwd_maxabs(got, ref, name):
    err = np.abs(got - ref).max()
    bound = 2e-2 * max(1.0, np.abs(ref).max())
    assert err <= bound, f"{name}: max abs err {err} > {bound}"


def _bwd_fro(got, ref, name, bound=BWD_REL_FRO):
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    assert rel <= bound, f"{name}: relative Frobenius err {rel}"
    print(f"{name}: rel Frobenius {rel:.3g}", flush=True)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c5"])
def test_full_size_sampled_parity(name):
    w = W.get(name)
    plan = PLAN[name]
    rng = np.random.default_rng(w.seed)
    res = _run(w)
    _check_inputs_match_cpu_draw(w, res, rng)
    segs = plan["segments"]
    if segs is None:
        segs = (w.scaled_segments[0], 1 if w.scaled_segments[0] != 1 else 2, w.num_segments - 1)
    dkdv_head = int(rng.integers(w.num_heads))
    scale = w.scale
    print(f"{name}: segments {segs}, all {w.num_heads} heads, dK/dV on head {dkdv_head}", flush=True)
    for s in segs:
        a, b = w.cu_seqlens_q[s], w.cu_seqlens_q[s + 1]
        shard = w.kind[s] == W.SHARD
        rng_ = _ranges(w, s)
        kidx = torch.cat([torch.arange(k0, k1, device="cuda") for k0, k1, _ in rng_])
        dq_got, dq_ref = [], []
        for h in range(w.num_heads):
            rows = _rows(rng, a, b)
            idx = torch.as_tensor(a + rows, device="cuda")
            qr, dor = _host(res["q"], idx, h), _host(res["do"], idx, h)
            ks = [_host(res["k"], slice(k0, k1), h) for k0, k1, _ in rng_]
            vs = [_host(res["v"], slice(k0, k1), h) for k0, k1, _ in rng_]
            kk, vv = np.concatenate(ks), np.concatenate(vs)
            # forward: per-block partials for shard rows, final output for every row
            if shard:
                for (k0, k1, b_), kb, vb in zip(rng_, ks, vs):
                    o_b, l_b = oracle.attend(qr, kb, vb, scale)
                    np.testing.assert_allclose(to64(res["parts"][0][b_, idx, h]), o_b, rtol=0, atol=O_TOL)
                    np.testing.assert_allclose(to64(res["parts"][1][b_, idx, h]), l_b, rtol=0, atol=LSE_TOL)
            o, l = oracle.attend(qr, kk, vv, scale)
            np.testing.assert_allclose(to64(res["out"][idx, h]), o, rtol=0, atol=O_TOL)
            np.testing.assert_allclose(to64(res["lse"][idx, h]), l, rtol=0, atol=LSE_TOL)
            # dQ of the sampled rows (needs only those rows' statistics)
            g_q, _, _ = oracle.attend_bwd(qr, kk, vv, dor, scale, k_rows=np.array([], dtype=np.int64))
            dq_got.append(to64(res["dq"][idx, h]))
            dq_ref.append(g_q)
            # one head, every query of the segment: forward and dQ on all rows,
            # dK/dV on sampled keys
            if h == dkdv_head and (not shard or plan["shard_dkdv"]):
                qa = _host(res["q"], slice(a, b), h)
                doa = _host(res["do"], slice(a, b), h)
                if shard:
                    for (k0, k1, b_), kb, vb in zip(rng_, ks, vs):
                        o_b, l_b = oracle.attend(qa, kb, vb, scale)
                        np.testing.assert_allclose(to64(res["parts"][0][b_, a:b, h]), o_b, rtol=0, atol=O_TOL)
                        np.testing.assert_allclose(to64(res["parts"][1][b_, a:b, h]), l_b, rtol=0, atol=LSE_TOL)
                o_all, l_all = oracle.attend(qa, kk, vv, scale)
                np.testing.assert_allclose(to64(res["out"][a:b, h]), o_all, rtol=0, atol=O_TOL)
                np.testing.assert_allclose(to64(res["lse"][a:b, h]), l_all, rtol=0, atol=LSE_TOL)
                keys = _rows(rng, 0, kk.shape[0], extra=10)
                g_qa, g_k, g_v = oracle.attend_bwd(qa, kk, vv, doa, scale, k_rows=keys)
                got_qa = to64(res["dq"][a:b, h])
                _bwd_maxabs(got_qa, g_qa, f"{name} seg {s} head {h} dq, all {b - a} rows")
                _bwd_fro(got_qa, g_qa, f"{name} seg {s} head {h} dq, all {b - a} rows", BWD_REL_FRO_POOLED)
                print(f"{name} seg {s} head {h}: forward and dQ checked on all {b - a} rows", flush=True)
                kp = kidx[torch.as_tensor(keys, device="cuda")]
                for got, ref, nm in ((to64(res["dk"][kp, h]), g_k, "dk"), (to64(res["dv"][kp, h]), g_v, "dv")):
                    _bwd_maxabs(got, ref, f"{name} seg {s} head {h} {nm}")
                    _bwd_fro(got, ref, f"{name} seg {s} head {h} {nm}")
        # dQ of the segment, all heads' sampled rows together: the max-abs bound takes its scale from the
        # whole sample (one head's two dozen rows of a nearly one-hot segment can miss its large entries)
        dq_got, dq_ref = np.concatenate(dq_got), np.concatenate(dq_ref)
        _bwd_maxabs(dq_got, dq_ref, f"{name} seg {s} all heads dq")
        _bwd_fro(dq_got, dq_ref, f"{name} seg {s} all heads dq", BWD_REL_FRO_POOLED)
        # identities that hold at any size, every head: sum_j dK_j = 0, sum_j dV_j = sum_i dO_i
        dk_sum = res["dk"][kidx].double().sum(0)
        dk_abs = res["dk"][kidx].double().abs().sum(0)
        assert (dk_sum.abs() <= 2e-2 * dk_abs + 1e-3).all(), f"{name} seg {s}: sum of dK not ~0"
        dv_sum = res["dv"][kidx].double().sum(0)
        do_sum = res["do"][a:b].double().sum(0)
        scale_ = res["dv"][kidx].double().abs().sum(0) + res["do"][a:b].double().abs().sum(0)
        assert ((dv_sum - do_sum).abs() <= 2e-2 * scale_ / np.sqrt(b - a) + 1e-2).all(), \
            f"{name} seg {s}: sum of dV != sum of dO"
    del res
    torch.cuda.empty_cache()
