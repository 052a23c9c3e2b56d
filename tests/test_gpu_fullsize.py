"""GPU parity at the benchmark's full sizes, in the launch configuration
bench.py times (one forward over the whole packed batch, the LSE merge, the
backward), checked on seeded samples the fp64 oracle computes one by one:

  * forward and dQ on sampled query rows (first, last, tile edges and seeded
    rows) of sampled segments and heads; a shard row is checked per block
    (partial O_b, LSE_b) and after the merge against attention over the
    concatenation of its blocks;
  * dK and dV on sampled keys of one head, which needs the oracle's O and LSE
    for every query of the segment; for the 31,110 x 497,760 shard this is
    too slow on the host, so there it is replaced by identities that hold at
    any size (sum over all keys of dK = 0, sum over all keys of dV = sum over
    queries of dO) checked on every head.

Inputs come from the seeded counter-based generator, drawn on the GPU for
the launch and re-drawn on the CPU (bit-identical) for the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_01150_amd import workloads as W
from tests._gpu import HAVE_GPU, api, to64

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="needs a GPU")]

O_TOL, LSE_TOL = 2e-2, 1e-3
# Backward: the gradients consume the forward output as stored (bf16), and
# D_i = dO_i . O_i inherits its rounding; for a nearly one-hot softmax
# (the x4-scaled segments) dS = P (dP - D) is a small difference, and the
# oracle alone shows a 0.55% relative dQ change from rounding O to bf16.
BWD_REL_FRO = 2e-2

# segments checked per workload, and whether dK/dV of the shard is sampled
PLAN = {
    "c2": dict(segments=(0, 7, 15), shard_dkdv=True),
    "c3": dict(segments=None, shard_dkdv=True),       # None: the scaled segment, a 3600 and the last 1560
    "c4": dict(segments=(0, 1, 6), shard_dkdv=True),
    "c5": dict(segments=(0, 1, 12), shard_dkdv=False),
}


def _run(w):
    dev = torch.device("cuda:0")
    desc = api.SegDesc.of(w)
    H, hd = w.num_heads, w.head_dim
    q, k, v, do = (w.full(t, device=dev) for t in (W.TENSOR_Q, W.TENSOR_K, W.TENSOR_V, W.TENSOR_DO))
    out, lse, o_part, lse_part = api.attn_fwd(desc, q, k, v, w.scale)
    parts = None
    if w.num_slots:
        # keep the per-block partials of the sampled rows before the merge overwrites nothing
        parts = (o_part, lse_part)
        api.lse_merge(desc, o_part, lse_part, out, lse)
    dq, dk, dv = api.attn_bwd(desc, q, k, v, out, lse, do, w.scale)
    torch.cuda.synchronize()
    del q, k, v
    return dict(out=out, lse=lse, parts=parts, dq=dq, dk=dk, dv=dv, do=do)


def _ranges(w, s):
    return [(w.cu_seqlens_k[j], w.cu_seqlens_k[j + 1], w.block_index[j])
            for j in range(w.kv_first[s], w.kv_first[s] + w.kv_count[s])]


def _rows(rng, a, b, extra=12):
    n = b - a
    base = {0, n - 1, min(n - 1, 127), min(n - 1, 128), min(n - 1, 63), min(n - 1, 64)}
    base |= set(rng.choice(n, size=min(n, extra), replace=False).tolist())
    return np.array(sorted(base), dtype=np.int64)


def _f64(t):
    return t.double().numpy()[:, 0]


def _check_bwd(got, ref, name):
    err = np.abs(got - ref).max()
    bound = 2e-2 * max(1.0, np.abs(ref).max())
    assert err <= bound, f"{name}: max abs err {err} > {bound}"
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    assert rel <= BWD_REL_FRO, f"{name}: relative Frobenius err {rel}"
    print(f"{name}: max abs {err:.3g} (bound {bound:.3g}), rel Frobenius {rel:.3g}")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c5"])
def test_full_size_sampled_parity(name):
    w = W.get(name)
    plan = PLAN[name]
    rng = np.random.default_rng(w.seed)
    res = _run(w)
    segs = plan["segments"]
    if segs is None:
        segs = (w.scaled_segments[0], 1 if w.scaled_segments[0] != 1 else 2, w.num_segments - 1)
    heads = sorted(rng.choice(w.num_heads, size=2, replace=False).tolist())
    scale = w.scale
    print(f"{name}: segments {segs} heads {heads}", flush=True)
    for s in segs:
        a, b = w.cu_seqlens_q[s], w.cu_seqlens_q[s + 1]
        rows = _rows(rng, a, b)
        shard = w.kind[s] == W.SHARD
        rng_ = _ranges(w, s)
        for hi, h in enumerate(heads):
            qr = np.concatenate([_f64(w.slice(W.TENSOR_Q, a + r, a + r + 1, heads=[h])) for r in rows])
            dor = np.concatenate([_f64(w.slice(W.TENSOR_DO, a + r, a + r + 1, heads=[h])) for r in rows])
            ks = [_f64(w.slice(W.TENSOR_K, k0, k1, heads=[h])) for k0, k1, _ in rng_]
            vs = [_f64(w.slice(W.TENSOR_V, k0, k1, heads=[h])) for k0, k1, _ in rng_]
            kk, vv = np.concatenate(ks), np.concatenate(vs)
            idx = torch.as_tensor(a + rows, device="cuda")
            # forward: per-block partials for shard rows, final output for every row
            if shard:
                for (k0, k1, b_), kb, vb in zip(rng_, ks, vs):
                    o_b, l_b = oracle.attend(qr, kb, vb, scale)
                    got_o = to64(res["parts"][0][b_, idx, h])
                    got_l = to64(res["parts"][1][b_, idx, h])
                    np.testing.assert_allclose(got_o, o_b, rtol=0, atol=O_TOL)
                    np.testing.assert_allclose(got_l, l_b, rtol=0, atol=LSE_TOL)
            o, l = oracle.attend(qr, kk, vv, scale)
            np.testing.assert_allclose(to64(res["out"][idx, h]), o, rtol=0, atol=O_TOL)
            np.testing.assert_allclose(to64(res["lse"][idx, h]), l, rtol=0, atol=LSE_TOL)
            # dQ of the sampled rows (needs only those rows' statistics)
            g_q, _, _ = oracle.attend_bwd(qr, kk, vv, dor, scale, k_rows=np.array([], dtype=np.int64))
            _check_bwd(to64(res["dq"][idx, h]), g_q, f"{name} seg {s} head {h} dq")
            # dK/dV of sampled keys: every query of the segment, first sampled head only
            if hi == 0 and (not shard or plan["shard_dkdv"]):
                qa = _f64(w.slice(W.TENSOR_Q, a, b, heads=[h]))
                doa = _f64(w.slice(W.TENSOR_DO, a, b, heads=[h]))
                keys = _rows(rng, 0, kk.shape[0], extra=10)
                _, g_k, g_v = oracle.attend_bwd(qa, kk, vv, doa, scale, q_rows=np.array([], dtype=np.int64),
                                                k_rows=keys)
                starts = np.concatenate([[0], np.cumsum([k1 - k0 for k0, k1, _ in rng_])])
                packed = np.array([rng_[np.searchsorted(starts, kj, side="right") - 1][0]
                                   + kj - starts[np.searchsorted(starts, kj, side="right") - 1] for kj in keys])
                kidx = torch.as_tensor(packed, device="cuda")
                _check_bwd(to64(res["dk"][kidx, h]), g_k, f"{name} seg {s} head {h} dk")
                _check_bwd(to64(res["dv"][kidx, h]), g_v, f"{name} seg {s} head {h} dv")
        # identities that hold at any size, every head: sum_j dK_j = 0, sum_j dV_j = sum_i dO_i
        kidx = torch.cat([torch.arange(k0, k1, device="cuda") for k0, k1, _ in rng_])
        dk_sum = res["dk"][kidx].double().sum(0)
        dk_abs = res["dk"][kidx].double().abs().sum(0)
        assert (dk_sum.abs() <= 2e-2 * dk_abs + 1e-3).all(), f"{name} seg {s}: sum of dK not ~0"
        dv_sum = res["dv"][kidx].double().sum(0)
        do_sum = res["do"][a:b].double().sum(0)
        scale_ = res["dv"][kidx].double().abs().sum(0) + res["do"][a:b].double().abs().sum(0)
        assert ((dv_sum - do_sum).abs() <= 2e-2 * scale_ / np.sqrt(b - a) + 1e-2).all(), \
            f"{name} seg {s}: sum of dV != sum of dO"
