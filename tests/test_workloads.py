"""Shapes and generator properties of the synthetic workloads."""
import os

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
