"""GPU test of the Ulysses (1,h,1) local staging (Sec. II-B, Tab. II; Sec.
IV-D's coalesced QKV-packed all-to-all): a group of ranks is simulated on
one device, the two all-to-alls being plain buffer reshuffles done here in
the test.  The layout kernels only move bytes, so they are checked bit for
bit: the unpacked head-subset Q/K/V against the full tensors, and the
local outputs after the inverse staging against one attention launch over
all heads (every head is computed by the same code either way).  The
attention itself is checked against the oracle."""
import numpy as np
import pytest
import torch

import oracle
from tests._gpu import HAVE_GPU, api, to64

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="needs a GPU")]


def _run(G, H, hd, shard_lens, seed):
    """shard_lens[j][s]: tokens of sequence s held by rank j (rank j's shard follows those of ranks < j)."""
    S = len(shard_lens[0])
    L = [sum(shard_lens[j][s] for j in range(G)) for s in range(S)]
    g = torch.Generator().manual_seed(seed)
    Qs, Ks, Vs = ([torch.randn((n, H, hd), generator=g).to(torch.bfloat16) for n in L] for _ in range(3))
    off = lambda j, s: sum(shard_lens[i][s] for i in range(j))
    local = lambda T, j: torch.cat([T[s][off(j, s):off(j, s) + shard_lens[j][s]] for s in range(S)]).cuda()
    cu_rank = np.array([np.concatenate([[0], np.cumsum(shard_lens[j])]) for j in range(G)], np.int32)
    Hl = H // G
    # pack on every rank, all-to-all by reshuffling
    sends = [api.ulysses_pack_qkv(G, local(Qs, j), local(Ks, j), local(Vs, j)) for j in range(G)]
    T = [int(cu_rank[j][-1]) for j in range(G)]
    full_q = torch.cat(Qs).cuda()
    full_k = torch.cat(Ks).cuda()
    full_v = torch.cat(Vs).cuda()
    cu = np.concatenate([[0], np.cumsum(L)]).astype(np.int32)
    desc_full = api.SegDesc(cu, np.zeros(S, np.uint8), np.arange(S, dtype=np.int32), np.ones(S, np.int32), cu,
                            np.zeros(S, np.int32), 0)
    out_full, lse_full, _, _ = api.attn_fwd(desc_full, full_q, full_k, full_v, 1.0 / hd ** 0.5)
    outs = []
    for r in range(G):
        recv = torch.cat([sends[j][r] for j in range(G)])                 # [T_full, Hl, 3, d], rank-major
        q, k, v = api.ulysses_unpack_qkv(G, cu_rank, recv, H)
        heads = slice(r * Hl, (r + 1) * Hl)
        assert torch.equal(q, full_q[:, heads]) and torch.equal(k, full_k[:, heads]) and torch.equal(v, full_v[:, heads])
        o, lse, _, _ = api.attn_fwd(desc_full, q, k, v, 1.0 / hd ** 0.5)
        outs.append(api.ulysses_pack_out(G, cu_rank, o, H))                  # rank-major [T_full, Hl, d]
    start = np.concatenate([[0], np.cumsum(T)])
    for j in range(G):
        recv = torch.stack([outs[r][start[j]:start[j + 1]] for r in range(G)])  # [G, T_j, Hl, d]
        got = api.ulysses_unpack_out(G, recv, H)
        torch.cuda.synchronize()
        rows = torch.cat([torch.arange(cu[s] + off(j, s), cu[s] + off(j, s) + shard_lens[j][s])
                          for s in range(S)]).long()
        assert torch.equal(got, out_full[rows.cuda()]), f"rank {j}: staged output differs from direct attention"
    # the attention itself against the oracle (one head per sequence)
    for s in range(S):
        if L[s] == 0:
            continue
        h = s % H
        o_ref, _ = oracle.attend(Qs[s][:, h].double().numpy(), Ks[s][:, h].double().numpy(),
                                 Vs[s][:, h].double().numpy(), 1.0 / hd ** 0.5)
        np.testing.assert_allclose(to64(out_full[cu[s]:cu[s + 1], h]), o_ref, rtol=0, atol=2e-2)


def test_ulysses_group4_uneven_shards():
    # three sequences, uneven shards, one rank with an empty shard of sequence 1
    _run(G=4, H=8, hd=128, shard_lens=((75, 20, 1), (75, 0, 0), (80, 37, 2), (70, 20, 1)), seed=41)


def test_ulysses_group2_d64():
    _run(G=2, H=6, hd=64, shard_lens=((128, 33), (129, 32)), seed=42)


def test_ulysses_group1_is_identity_layout():
    _run(G=1, H=4, hd=128, shard_lens=((100, 7),), seed=43)
