"""The backward's own error, apart from the forward's.

zl_attn_bwd is fed an O and LSE computed by the oracle (the final output of
every row rounded once to bf16, its LSE rounded to fp32) in place of the GPU
forward's, and its gradients are compared with the oracle's backward on that
same stored O and LSE (oracle.attend_bwd_given).  No GPU forward enters the
comparison, so what remains is the backward's own rounding: P and dS as bf16
MFMA operands and bf16 outputs, 0.25% in the CPU error budget
(tests/test_bwd_error_budget.py).  Bound: max abs error <= 1e-2 * max(1,
max|ref|) and relative Frobenius error <= 1e-2, on small packed batches (a
x4-scaled segment among them) and on the x4-scaled 32,760-token video of the
mixed image-video batch at full size.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_01150_amd import workloads as W
from tests import _descs
from tests._gpu import HAVE_GPU, api, to64

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="needs a GPU")]

BWD_ISO = 1e-2


def _check(got, ref, name):
    err = np.abs(got - ref).max()
    bound = BWD_ISO * max(1.0, np.abs(ref).max())
    assert err <= bound, f"{name}: max abs err {err} > {bound}"
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    assert rel <= BWD_ISO, f"{name}: relative Frobenius err {rel}"
    print(f"{name}: max abs {err:.3g}, rel Frobenius {rel:.3g}", flush=True)


def _stored(o, lse):
    """The oracle's O and LSE as a forward would store them (bf16, fp32), in fp64 and as torch tensors."""
    ob = torch.from_numpy(np.ascontiguousarray(o, dtype=np.float32)).to(torch.bfloat16)
    lb = torch.from_numpy(np.ascontiguousarray(lse, dtype=np.float32))
    return ob, lb, ob.double().numpy(), lb.double().numpy()


def _segments(d):
    for s in range(len(d["kind"])):
        r0, r1 = d["cu_seqlens_q"][s], d["cu_seqlens_q"][s + 1]
        j0 = d["kv_first"][s]
        bounds = [(d["cu_seqlens_k"][j], d["cu_seqlens_k"][j + 1]) for j in range(j0, j0 + d["kv_count"][s])]
        yield r0, r1, bounds


def _small(d, H, hd, seed, scaled_segments=()):
    g = torch.Generator().manual_seed(seed)
    tq, tk = d["cu_seqlens_q"][-1], d["cu_seqlens_k"][-1]
    q, k, v, do = (torch.randn((n, H, hd), generator=g).to(torch.bfloat16) for n in (tq, tk, tk, tq))
    for s in scaled_segments:   # x4 is exact in bf16
        r0, r1, bounds = list(_segments(d))[s]
        q[r0:r1] *= 4
        for a, b in bounds:
            k[a:b] *= 4
    scale = hd ** -0.5
    q64, k64, v64, do64 = (t.double().numpy() for t in (q, k, v, do))
    ref = oracle.packed_forward(d, q64, k64, v64, scale)
    o_t, l_t, o_in, l_in = _stored(np.nan_to_num(ref["final_out"]), np.nan_to_num(ref["final_lse"]))
    desc = api.SegDesc.of(d)
    dq, dk, dv = api.attn_bwd(desc, q.cuda(), k.cuda(), v.cuda(), o_t.cuda(), l_t.cuda(), do.cuda(), scale)
    torch.cuda.synchronize()
    rq, rk, rv = np.zeros_like(q64), np.zeros_like(k64), np.zeros_like(v64)
    for r0, r1, bounds in _segments(d):
        if r1 == r0:
            continue
        for h in range(H):
            kk = np.concatenate([k64[a:b, h] for a, b in bounds])
            vv = np.concatenate([v64[a:b, h] for a, b in bounds])
            gq, gk, gv = oracle.attend_bwd_given(q64[r0:r1, h], kk, vv, do64[r0:r1, h], o_in[r0:r1, h],
                                                 l_in[r0:r1, h], scale)
            rq[r0:r1, h] = gq
            off = 0
            for a, b in bounds:
                rk[a:b, h] += gk[off:off + b - a]
                rv[a:b, h] += gv[off:off + b - a]
                off += b - a
    for got, ref_, nm in ((dq, rq, "dq"), (dk, rk, "dk"), (dv, rv, "dv")):
        _check(to64(got), ref_, nm)


@pytest.mark.parametrize("hd", [64, 128])
def test_backward_alone_mixed_batch(hd):
    # whole 200, empty whole, whole 77, a 150-query shard on blocks of 300/0/129 keys, a 33-query shard
    _small(_descs.mixed_small(), 3, hd, 90 + hd)


def test_backward_alone_scaled_segment():
    """A x4-scaled whole segment (Q and K times 4: a nearly one-hot softmax) beside an unscaled shard."""
    d = _descs.desc(cu_q=(0, 300, 500), kind=(0, 1), kv_first=(0, 1), kv_count=(1, 3),
                    cu_k=(0, 300, 429, 493, 700), block_index=(0, 2, 0, 1), num_slots=3)
    _small(d, 2, 128, 93, scaled_segments=(0,))


@pytest.mark.timeout(900)
def test_backward_alone_scaled_video_full_size():
    """The x4-scaled 32,760-token video of the mixed image-video batch, full size: one seeded head's O and
    LSE for every video row come from the oracle (rounded as stored) and replace the GPU forward's for that
    head; the backward runs on the whole batch; dQ is checked on 64 sampled rows and dK/dV on 24 sampled
    keys of that head against the oracle's backward on the same stored O and LSE."""
    w = W.get("c3")
    s = w.scaled_segments[0]
    a, b = w.cu_seqlens_q[s], w.cu_seqlens_q[s + 1]
    k0, k1 = w.cu_seqlens_k[w.kv_first[s]], w.cu_seqlens_k[w.kv_first[s] + 1]
    rng = np.random.default_rng(w.seed + 7)
    h = int(rng.integers(w.num_heads))
    dev = torch.device("cuda:0")
    desc = api.SegDesc.of(w)
    q, k, v, do = (w.full(t, device=dev) for t in (W.TENSOR_Q, W.TENSOR_K, W.TENSOR_V, W.TENSOR_DO))
    for t, x, r in ((W.TENSOR_Q, q, a), (W.TENSOR_K, k, k0), (W.TENSOR_V, v, k1 - 1), (W.TENSOR_DO, do, b - 1)):
        assert torch.equal(x[r:r + 1].cpu(), w.slice(t, r, r + 1))   # device draw == CPU draw
    out, lse, _, _ = api.attn_fwd(desc, q, k, v, w.scale)
    host = lambda t, sl: t[sl, h].double().cpu().numpy()
    qa, doa = host(q, slice(a, b)), host(do, slice(a, b))
    kk, vv = host(k, slice(k0, k1)), host(v, slice(k0, k1))
    print(f"head {h}: oracle forward of {b - a} rows", flush=True)
    o, l = oracle.attend(qa, kk, vv, w.scale)
    o_t, l_t, o_in, l_in = _stored(o, l)
    out[a:b, h] = o_t.to(dev)
    lse[a:b, h] = l_t.to(dev)
    dq, dk, dv = api.attn_bwd(desc, q, k, v, out, lse, do, w.scale)
    torch.cuda.synchronize()
    rows = np.sort(rng.choice(b - a, size=64, replace=False))
    none = np.array([], dtype=np.int64)
    gq, _, _ = oracle.attend_bwd_given(qa[rows], kk, vv, doa[rows], o_in[rows], l_in[rows], w.scale, k_rows=none)
    _check(to64(dq[torch.as_tensor(a + rows, device=dev), h]), gq, f"video head {h} dq")
    keys = np.sort(rng.choice(k1 - k0, size=24, replace=False))
    _, gk, gv = oracle.attend_bwd_given(qa, kk, vv, doa, o_in, l_in, w.scale, q_rows=none, k_rows=keys)
    kidx = torch.as_tensor(k0 + keys, device=dev)
    _check(to64(dk[kidx, h]), gk, f"video head {h} dk")
    _check(to64(dv[kidx, h]), gv, f"video head {h} dv")
