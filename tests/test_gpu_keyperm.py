"""Key-permutation invariance on the device.

Softmax attention sums over a segment's keys, so permuting the rows of K and
V jointly inside a segment must leave that segment's O and LSE unchanged (up
to rounding: the kernels add in a different order and their lazy rescaling
triggers at other keys), must permute its dK and dV rows the same way and
leave its dQ unchanged, and must not touch any other segment at all: every
other segment's outputs and gradients stay equal bit for bit (Sec. IV-D: one
block-diagonal call keeps sequences separate).  Checked on a small packed
batch (a whole segment and a shard whose blocks are each permuted) and on the
full-size mixed image-video batch with the 32,760-token video's keys
permuted.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_01150_amd import workloads as W
from tests import _descs
from tests._gpu import HAVE_GPU, api, to64

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="needs a GPU")]

# Each run is within the oracle bounds (2e-2 on O, 1e-3 on LSE) of the same exact values, so two runs
# may differ by twice that (at |O| near 3.5, one bf16 ulp is 0.0156 and the runs can round apart).  The
# permuted run's sampled rows are also checked against the oracle at the single bounds.
O_TOL, LSE_TOL, REL = 2e-2, 1e-3, 2e-2


def _path(desc, q, k, v, do, scale):
    out, lse, o_part, lse_part = api.attn_fwd(desc, q, k, v, scale)
    if desc.num_slots:
        api.lse_merge(desc, o_part, lse_part, out, lse)
    dq, dk, dv = api.attn_bwd(desc, q, k, v, out, lse, do, scale)
    torch.cuda.synchronize()
    return dict(out=out, lse=lse, dq=dq, dk=dk, dv=dv, o_part=o_part, lse_part=lse_part)


def _rel(a, b):
    a, b = to64(a), to64(b)
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30)


def _compare(ref, got, perm_rows, q_rows, key_index, slots=()):
    """perm_rows: packed K/V rows that were permuted; key_index: for each of them, the row of the
    unpermuted batch it came from; q_rows: query rows of the permuted segment."""
    dev = ref["out"].device
    qi = torch.as_tensor(q_rows, device=dev)
    other_q = torch.ones(ref["out"].shape[0], dtype=torch.bool, device=dev)
    other_q[qi] = False
    other_k = torch.ones(ref["dk"].shape[0], dtype=torch.bool, device=dev)
    other_k[torch.as_tensor(perm_rows, device=dev)] = False
    for name, sel in (("out", other_q), ("lse", other_q), ("dq", other_q), ("dk", other_k), ("dv", other_k)):
        assert torch.equal(got[name][sel], ref[name][sel]), f"{name} of another segment changed"
    assert (got["out"][qi].float() - ref["out"][qi].float()).abs().max().item() <= 2 * O_TOL
    assert (got["lse"][qi] - ref["lse"][qi]).abs().max().item() <= 2 * LSE_TOL
    for b in slots:   # per-block partials of a shard whose blocks were each permuted
        assert (got["o_part"][b][qi] - ref["o_part"][b][qi]).abs().max().item() <= 2 * O_TOL
        dl = torch.nan_to_num(got["lse_part"][b][qi] - ref["lse_part"][b][qi], nan=0.0)  # an empty block: -inf both
        assert dl.abs().max().item() <= 2 * LSE_TOL
    assert _rel(got["dq"][qi], ref["dq"][qi]) <= REL
    pr = torch.as_tensor(perm_rows, device=dev)
    src = torch.as_tensor(key_index, device=dev)
    assert _rel(got["dk"][pr], ref["dk"][src]) <= REL
    assert _rel(got["dv"][pr], ref["dv"][src]) <= REL


def test_key_permutation_small_batch():
    d = _descs.mixed_small()   # seg 0: whole 200; seg 3: a 150-query shard on blocks of 300 / 0 / 129 keys
    H, hd = 2, 128
    desc = api.SegDesc.of(d)
    g = torch.Generator().manual_seed(81)
    tq, tk = d["cu_seqlens_q"][-1], d["cu_seqlens_k"][-1]
    q, k, v, do = (torch.randn((n, H, hd), generator=g).to(torch.bfloat16).cuda() for n in (tq, tk, tk, tq))
    scale = hd ** -0.5
    ref = _path(desc, q, k, v, do, scale)
    rng = np.random.default_rng(82)
    for s in (0, 3):
        rows, src = [], []
        for j in range(d["kv_first"][s], d["kv_first"][s] + d["kv_count"][s]):
            a, b = d["cu_seqlens_k"][j], d["cu_seqlens_k"][j + 1]
            rows += list(range(a, b))
            src += (a + rng.permutation(b - a)).tolist()
        k2, v2 = k.clone(), v.clone()
        idx, sidx = torch.as_tensor(rows, device="cuda"), torch.as_tensor(src, device="cuda")
        k2[idx], v2[idx] = k[sidx], v[sidx]
        got = _path(desc, q, k2, v2, do, scale)
        slots = [d["block_index"][j] for j in range(d["kv_first"][s], d["kv_first"][s] + d["kv_count"][s])] \
            if d["kind"][s] == 1 else []
        _compare(ref, got, rows, np.arange(d["cu_seqlens_q"][s], d["cu_seqlens_q"][s + 1]), src, slots)


@pytest.mark.timeout(600)
def test_key_permutation_full_size_video():
    w = W.get("c3")
    s = 0 if w.kind[0] == W.WHOLE and w.cu_seqlens_q[1] == 32760 else None
    assert s is not None, "the mixed batch's first segment is the 32,760-token video"
    dev = torch.device("cuda:0")
    desc = api.SegDesc.of(w)
    q, k, v, do = (w.full(t, device=dev) for t in (W.TENSOR_Q, W.TENSOR_K, W.TENSOR_V, W.TENSOR_DO))
    ref = _path(desc, q, k, v, do, w.scale)
    k0, k1 = w.cu_seqlens_k[w.kv_first[s]], w.cu_seqlens_k[w.kv_first[s] + 1]
    perm = np.random.default_rng(83).permutation(k1 - k0)
    rows = np.arange(k0, k1)
    src = k0 + perm
    idx = torch.as_tensor(src, device=dev)
    k[k0:k1] = k[idx].clone()
    v[k0:k1] = v[idx].clone()
    got = _path(desc, q, k, v, do, w.scale)
    _compare(ref, got, rows, np.arange(w.cu_seqlens_q[s], w.cu_seqlens_q[s + 1]), src)
    # the permuted run against the oracle on sampled rows of two heads
    rng = np.random.default_rng(84)
    qr = np.sort(rng.choice(w.cu_seqlens_q[s + 1] - w.cu_seqlens_q[s], size=32, replace=False)) + w.cu_seqlens_q[s]
    qi = torch.as_tensor(qr, device=dev)
    for h in rng.choice(w.num_heads, size=2, replace=False):
        kk = k[k0:k1, h].double().cpu().numpy()
        vv = v[k0:k1, h].double().cpu().numpy()
        o, l = oracle.attend(q[qi, h].double().cpu().numpy(), kk, vv, w.scale)
        np.testing.assert_allclose(to64(got["out"][qi, h]), o, rtol=0, atol=O_TOL)
        np.testing.assert_allclose(to64(got["lse"][qi, h]), l, rtol=0, atol=LSE_TOL)
