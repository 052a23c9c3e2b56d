"""The bucket catalog, the synthetic batches and the planning glue of the
price-table tool (CPU), and one small price measurement (GPU)."""
import math

import numpy as np
import pytest
import torch

from paper_2608_01150_amd import api
from paper_2608_01150_amd import price_table as PT
from paper_2608_01150_amd import workloads as W


def test_catalog_matches_wan_token_counts():
    # Sec. I: a 15 s 1080p video is 497,760 tokens; the benchmark shapes use 1560 / 3600 / 32,760 / 75,600
    assert W.CATALOG["vid1080-15s"] == 497_760
    assert W.CATALOG["img480"] == 1560 and W.CATALOG["img720"] == 3600
    assert W.CATALOG["vid480-5s"] == 32_760 and W.CATALOG["vid720-5s"] == 75_600
    assert W.latent_frames(5) == 21 and W.latent_frames(15) == 61
    assert sorted(W.CATALOG.values()) == sorted(set(W.CATALOG.values()))


@pytest.mark.parametrize("seed,share,sec", [(1, 0.35, 10), (2, 0.6, 10), (3, 0.5, 15), (4, 0.05, 15)])
def test_synthetic_batch_budget_and_share(seed, share, sec):
    N, budget = 8, 350_000
    b = W.synthetic_batch(N, budget, share, sec, seed)
    toks = [W.CATALOG[x] for x in b]
    vid = [W.CATALOG[x] for x in b if x.startswith("vid")]
    assert sum(toks) <= N * budget
    assert sum(toks) > N * budget - max(W.CATALOG[i] for i in W.IMAGE_BUCKETS)
    assert len(vid) >= 1 and all(x.endswith(f"-{sec}s") for x in b if x.startswith("vid"))
    assert sum(vid) <= share * N * budget or len(vid) == 1
    assert b == W.synthetic_batch(N, budget, share, sec, seed)


def test_even_split_and_config_segments():
    assert PT.even_split(10, 4) == [3, 3, 2, 2]
    assert PT.config_segments(10, "ring-4") == [("shard", 3, 0, [(3, 0, 0), (3, 3, 1), (2, 6, 2), (2, 8, 3)])]
    assert PT.config_segments(10, "gather-4") == [("shard", 3, 0, [(10, 0, 0)])]
    assert PT.config_segments(10, "whole") == PT.config_segments(10, "ulysses-2") == [("whole", 10, 0)]
    assert PT.configs_for("img480", 12, [2, 4, 8]) == ["whole"]
    assert "ulysses-8" not in PT.configs_for("vid480-5s", 12, [2, 4, 8])


def _model_prices(H=12):
    P = {"heads": H, "head_dim": 128, "prices": {}}
    for b, L in W.CATALOG.items():
        e = {"tokens": L, "whole": L * L * 1e-8 + L * 1e-4}
        for k in (2, 4, 8, 16):
            e[f"ring-{k}"] = e["whole"] / k * 1.05
        P["prices"][b] = e
    return P


@pytest.mark.parametrize("g", [1, 2, 4, 8])
@pytest.mark.parametrize("rule", ["eq8", "tokens"])
def test_plan_ledgers_and_rank_descriptors(g, rule):
    N = 8
    P = _model_prices()
    batch = W.synthetic_batch(N, 120_000, 0.4, 10, 11)
    placed, per_rank, load, mem, floor = PT.plan(batch, P, N, g, 150e3, 1e15, rule)
    cfg = "whole" if g == 1 else f"ring-{g}"
    fillers = [b for b in batch if not b.startswith("vid")]
    assert sorted(sum(per_rank, [])) == sorted(fillers)
    assert math.isclose(sum(load), sum(P["prices"][b][cfg] * g for b, _ in placed)
                        + sum(P["prices"][b]["whole"] for b in fillers), rel_tol=1e-12)
    assert math.isclose(floor, sum(P["prices"][b]["whole"] for b in batch) / N, rel_tol=1e-12)
    tokens = 0
    for r in range(N):
        segs = PT.rank_segments(placed, per_rank[r], g, r)
        w = W.build_segments("r", 2, 64, segs, 1)
        items, _ = api.plan_dump(api.SegDesc.of(w), 2, 64, torch.bfloat16, api.ZL_OP_BWD)   # validates
        assert items.shape[0] > 0 or not segs
        tokens += w.total_q
    assert tokens == sum(W.CATALOG[b] for b in batch)      # every token of the batch is some rank's query row


@pytest.mark.gpu
def test_price_measurement_small():
    dev = torch.device("cuda:0")
    out = {}
    for b, c in [("img256", "whole"), ("vid480-5s", "ring-2"), ("vid480-5s", "gather-2"),
                 ("vid480-5s", "ulysses-2")]:
        ms, copies = PT.price_one(b, c, 2, 128, dev)
        print(f"{b} {c}: {ms:.4f} ms (x{copies})", flush=True)
        assert math.isfinite(ms) and ms > 0
        out[c] = ms
    # ring-2 and gather-2 do the same MFMA work per rank (half the queries against all keys)
    assert 0.5 < out["ring-2"] / out["gather-2"] < 2.0
