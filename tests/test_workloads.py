"""Shapes and generator properties of the synthetic workloads."""
import os

import numpy as np
import torch

from paper_2608_01150_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "wan_tokens.txt")


def _golden():
    vals = {}
    for line in open(GOLDEN):
        if line.strip() and not line.startswith("#"):
            name, value = line.split()[:2]
            vals[name] = int(value)
    return vals


def test_token_arithmetic_matches_paper():
    g = _golden()
    c5 = W.get("c5")
    # one GPU's share at CP=16 is 1/16 of the 15 s 1080p video
    assert 16 * (c5.cu_seqlens_q[1] - c5.cu_seqlens_q[0]) == g["video_1080p_15s"]
    assert c5.cu_seqlens_k[16] == g["video_1080p_15s"]
    c4 = W.get("c4")
    assert c4.cu_seqlens_k[8] == g["video_720p_81f"]
    c3 = W.get("c3")
    lens = [c3.cu_seqlens_q[s + 1] - c3.cu_seqlens_q[s] for s in range(c3.num_segments)]
    assert lens == [g["video_480p_81f"]] + [g["image_720x1280"]] * 2 + [g["image_480x832"]] * 8


def test_pair_counts():
    expect = {"c1": 151552, "c2": 38937600, "c3": 1118606400, "c4": 729021600, "c5": 15556622400}
    for name, pairs in expect.items():
        assert W.get(name).pair_count() == pairs


def test_slices_are_consistent_and_seeded():
    w = W.get("c2")
    full = w.slice(W.TENSOR_K, 100, 140)
    part = w.slice(W.TENSOR_K, 120, 130, heads=[3, 7])
    assert torch.equal(full[20:30][:, [3, 7]], part)
    assert not torch.equal(w.slice(W.TENSOR_Q, 0, 8), w.slice(W.TENSOR_K, 0, 8))
    x = w.slice(W.TENSOR_V, 0, 4000).float()
    assert abs(x.mean().item()) < 0.01 and abs(x.std().item() - 1) < 0.01


def test_scaled_segment_is_exactly_times_four():
    w = W.get("c3")
    (s,) = w.scaled_segments
    a, b = w.rows_of_segment_q(s)
    plain = W.draw(w.seed, W.TENSOR_Q, torch.arange(a * w.num_heads * w.head_dim,
                                                      (a + 2) * w.num_heads * w.head_dim), torch.bfloat16)
    got = w.slice(W.TENSOR_Q, a, a + 2).reshape(-1)
    assert torch.equal(got, plain * 4)


def test_draw_follows_the_standard_normal():
    """The quantile-table generator against N(0,1): moments, tail fractions at 2, 3 and 4 sigma,
    the Kolmogorov-Smirnov distance on 2^21 fp32 draws, the sign symmetry of its table, and the
    bound of about 5.06 sigma set by the quarter-bin outer edges."""
    from scipy.special import ndtr, ndtri
    n = 1 << 21
    x = W.draw(7, 0, torch.arange(n, dtype=torch.int64), dtype=torch.float32).double().numpy()
    assert abs(x.mean()) < 3e-3 and abs(x.std() - 1) < 3e-3
    assert abs(((x - x.mean()) ** 4).mean() / x.var() ** 2 - 3) < 0.03
    for t in (2.0, 3.0, 4.0):
        want = 2 * ndtr(-t)
        got = (np.abs(x) > t).mean()
        assert abs(got - want) < 5 * np.sqrt(want / n), (t, got, want)
    xs = np.sort(x)
    cdf = ndtr(xs)
    ks = max((np.arange(1, n + 1) / n - cdf).max(), (cdf - np.arange(n) / n).max())
    assert ks < 1.63 / np.sqrt(n)          # 1% level of the KS test
    e = W._normal_edges("cpu").double().numpy()
    assert np.array_equal(e, -e[::-1])
    assert e[-1] == np.float32(ndtri(1 - 0.25 / (1 << W._QBITS)))
    assert np.abs(x).max() <= e[-1] and 5.0 < e[-1] < 5.1
