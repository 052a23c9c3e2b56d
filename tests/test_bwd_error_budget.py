"""Error budget of the bf16 backward, term by term, on the CPU.

The GPU backward differs from the exact fp64 gradients through three
roundings, each emulated here with numpy on top of the oracle's definitions
(no GPU code is involved):

  O storage     the forward's output is stored as bf16, and D_i = dO_i . O_i
                reads it back;
  forward P     the forward rounds each P_ij to bf16 before O += P V and
                normalises by the sum of the rounded values (the LSE takes
                the unrounded sum), so the stored O carries that error too;
  backward P/dS the backward rounds P_ij (for dV) and dS_ij (for dK, dQ) to
                bf16 before the MFMAs, and stores dQ, dK, dV as bf16.

Each term is reported as the relative Frobenius error of dQ, dK, dV against
the exact backward, on unscaled inputs and on the x4-scaled video segment of
the mixed image-video batch (Q and K times 4: a nearly one-hot softmax, where
dS = P (dP - D) is a small difference of nearly equal terms and the error of D
counts most).  The asserts tie the two GPU tolerances to these numbers:

  * the backward alone (O and LSE given, as the isolated GPU test feeds them)
    must stay well inside its 1e-2 bound;
  * the end-to-end chain (forward P, O storage, backward P/dS) must stay
    inside the 2e-2 bound of the tests that run the GPU forward first.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_01150_amd import workloads as W


def bf16(x):
    """Round to bf16 (nearest even) and back to fp64."""
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).double().numpy()


def fp32(x):
    return np.asarray(x, dtype=np.float32).astype(np.float64)


def rel(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def forward_emulated(q, k, v, scale):
    """O as the bf16 forward stores it: P rounded to bf16 in the P V product and in the row sum that
    normalises it, the result rounded to bf16; LSE from the unrounded row sum, rounded to fp32."""
    s = scale * (q @ k.T)
    m = s.max(axis=1, keepdims=True)
    p = np.exp(s - m)
    l = p.sum(axis=1, keepdims=True)
    pb = bf16(p)
    o = bf16((pb @ v) / pb.sum(axis=1, keepdims=True))
    lse = fp32(m[:, 0] + np.log(l[:, 0]))
    return o, lse


def backward_emulated(q, k, v, do, o, lse, scale, rows=None):
    """The bf16 backward on a given O and LSE: D in full precision from the given O, P and dS rounded
    to bf16 where they enter the products, outputs rounded to bf16.  rows: dQ of those rows only."""
    dsum = (do * o).sum(axis=1)
    s = scale * (q @ k.T)
    p = np.exp(s - lse[:, None])
    ds = p * (do @ v.T - dsum[:, None])
    pb, dsb = bf16(p), bf16(ds)
    if rows is not None:
        return bf16(scale * (dsb[rows] @ k)), None, None
    return bf16(scale * (dsb @ k)), bf16(scale * (dsb.T @ q)), bf16(pb.T @ do)


def _case(scaled, n=1024, d=128, seed=7):
    g = torch.Generator().manual_seed(seed)
    q, k, v, do = (torch.randn((n, d), generator=g).to(torch.bfloat16).double().numpy() for _ in range(4))
    if scaled:
        q, k = 4 * q, 4 * k
    return q, k, v, do


def budget(q, k, v, do, scale):
    exact = oracle.attend_bwd(q, k, v, do, scale)
    o, lse = oracle.attend(q, k, v, scale)
    o_store = bf16(o)
    o_fwd, lse_fwd = forward_emulated(q, k, v, scale)
    terms = {
        "O storage": oracle.attend_bwd_given(q, k, v, do, o_store, lse, scale),
        "forward P + O storage": oracle.attend_bwd_given(q, k, v, do, o_fwd, lse_fwd, scale),
        "backward P/dS + outputs": backward_emulated(q, k, v, do, o, fp32(lse), scale),
        "end to end": backward_emulated(q, k, v, do, o_fwd, lse_fwd, scale),
    }
    return {name: [rel(g, e) for g, e in zip(got, exact)] for name, got in terms.items()}


@pytest.mark.parametrize("scaled", [False, True])
def test_backward_error_budget(scaled):
    q, k, v, do = _case(scaled)
    b = budget(q, k, v, do, 128 ** -0.5)
    for name, (eq, ek, ev) in b.items():
        print(f"{'x4' if scaled else 'x1'} {name:24s} dq {eq:.2e} dk {ek:.2e} dv {ev:.2e}")
    # the backward on its own (what the isolated GPU test compares against its 1e-2 bound)
    assert max(b["backward P/dS + outputs"]) <= 0.5e-2
    # the whole chain (what the end-to-end tests compare against their 2e-2 bound)
    assert max(b["end to end"]) <= 1.5e-2


def test_video_segment_dq_budget():
    """The same chain on the mixed batch's actual x4-scaled video (32,760 keys), on 256 query rows of
    head 19: dQ needs only those rows' O and LSE, so the full key length is affordable here.

    On such a segment a few rows carry most of dQ's norm (a nearly one-hot row has dQ close to 0 and a
    relative error near 1), so a relative Frobenius error taken over a small row sample spreads widely
    around the segment's value.  The spread over random subsets is what a sampled GPU check sees: at 18
    rows (the sample of the earlier full-size test) its upper tail reaches past 1%, the size of the
    largest value the GPU showed there; at 64 rows it stays under 1.2%."""
    w = W.get("c3")
    s = w.scaled_segments[0]
    a, b = w.cu_seqlens_q[s], w.cu_seqlens_q[s + 1]
    k0, k1 = w.cu_seqlens_k[w.kv_first[s]], w.cu_seqlens_k[w.kv_first[s] + 1]
    h = 19
    rng = np.random.default_rng(30)
    rows = np.sort(rng.choice(b - a, size=256, replace=False))
    f = lambda t, r0, r1: w.slice(t, r0, r1, heads=[h]).double().numpy()[:, 0]
    q = np.concatenate([f(W.TENSOR_Q, a + r, a + r + 1) for r in rows])
    do = np.concatenate([f(W.TENSOR_DO, a + r, a + r + 1) for r in rows])
    k, v = f(W.TENSOR_K, k0, k1), f(W.TENSOR_V, k0, k1)
    scale = w.scale
    none = np.array([], dtype=np.int64)
    exact, _, _ = oracle.attend_bwd(q, k, v, do, scale, k_rows=none)
    o, lse = oracle.attend(q, k, v, scale)
    o_fwd, lse_fwd = forward_emulated(q, k, v, scale)
    res = {
        "O storage": oracle.attend_bwd_given(q, k, v, do, bf16(o), lse, scale, k_rows=none)[0],
        "forward P + O storage": oracle.attend_bwd_given(q, k, v, do, o_fwd, lse_fwd, scale, k_rows=none)[0],
        "backward P/dS + outputs": backward_emulated(q, k, v, do, o, fp32(lse), scale, rows=slice(None))[0],
        "end to end": backward_emulated(q, k, v, do, o_fwd, lse_fwd, scale, rows=slice(None))[0],
    }
    errs = {name: rel(g, exact) for name, g in res.items()}
    for name, e in errs.items():
        print(f"video x4 head {h} {name:24s} dq {e:.2e}")
    assert errs["backward P/dS + outputs"] <= 0.5e-2
    assert errs["end to end"] <= 1e-2
    e2e = res["end to end"]
    pick = np.random.default_rng(1)
    tails = {}
    for n in (18, 64):
        vals = [rel(e2e[sub], exact[sub]) for sub in (pick.choice(len(rows), size=n, replace=False)
                                                    for _ in range(2000))]
        tails[n] = np.percentile(vals, 99.9)
        print(f"  end to end over {n}-row subsets: median {np.median(vals):.2e} p99 {np.percentile(vals, 99):.2e} "
              f"p99.9 {tails[n]:.2e}")
    assert tails[18] > 1e-2          # small samples do reach the values seen on the GPU
    assert tails[18] <= 2e-2 and tails[64] <= 1.2e-2
    # The largest element error against max|ref| as the scale: taken over these 256 rows it stays well
    # inside 2e-2; taken over a two-dozen-row sample, whose max|ref| can miss the segment's large
    # entries, it spreads up to about 2% (which is why the full-size test pools a segment's sampled
    # rows over all heads before taking the scale).
    err = np.abs(e2e - exact).max(axis=1)
    scale_all = max(1.0, np.abs(exact).max())
    assert err.max() / scale_all <= 1e-2
    ratios = []
    for sub in (pick.choice(len(rows), size=24, replace=False) for _ in range(2000)):
        ratios.append(err[sub].max() / max(1.0, np.abs(exact[sub]).max()))
    print(f"  largest element error / max|ref|: {err.max() / scale_all:.2e} over 256 rows, "
          f"p99.9 {np.percentile(ratios, 99.9):.2e} over 24-row samples")
