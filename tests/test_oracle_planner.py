"""Pins for the oracle's Filler Packing (Sec. IV-C, Eq. 8).

Eq. 8 is a greedy rule, so it is pinned by the textbook rules it reduces to
when one resource cannot bind, by Graham's bound on one of them, by two
hand-worked cases where the two resources disagree, and by invariants
(scale invariance of the normalised slacks, memory feasibility).
"""
import heapq
import itertools
import random

import pytest

import oracle


def _lpt(price, load0):
    """Graham's LPT, written independently: jobs by decreasing size (stable),
    each to the least-loaded machine (lowest index on ties)."""
    heap = [(float(c), r) for r, c in enumerate(load0)]
    heapq.heapify(heap)
    rank_of = [-1] * len(price)
    for s in sorted(range(len(price)), key=lambda s: (-price[s], s)):
        c, r = heapq.heappop(heap)
        rank_of[s] = r
        heapq.heappush(heap, (c + price[s], r))
    return rank_of


def _worst_fit(need, free):
    """Worst fit in input order: each item to the bin with the most free
    space that still holds it (lowest index on ties); None where it fails."""
    free = list(free)
    rank_of = []
    for s, x in enumerate(need):
        cand = [r for r in range(len(free)) if free[r] >= x]
        if not cand:
            return rank_of, s
        r = max(cand, key=lambda r: (free[r], -r))
        free[r] -= x
        rank_of.append(r)
    return rank_of, None


def test_load_floor():
    assert oracle.load_floor([1.0, 2.0, 3.0, 6.0], 4) == 3.0
    assert oracle.load_floor([5], 2) == 2.5


@pytest.mark.parametrize("seed", range(12))
def test_reduces_to_lpt_when_memory_is_free(seed):
    """No memory demand: rho^M = 1 >= rho^C, so Eq. 8 maximises the compute
    slack, i.e. picks the least-loaded rank: LPT from the anchor loads."""
    rng = random.Random(seed)
    n_ranks = rng.randint(2, 8)
    n = rng.randint(1, 40)
    price = [float(rng.randint(1, 9)) for _ in range(n)]          # duplicates on purpose
    load0 = [float(rng.choice([0, 0, rng.randint(0, 30)])) for _ in range(n_ranks)]
    mem = [[0.0] * n_ranks for _ in range(n)]
    F = oracle.load_floor(price + load0, n_ranks)
    rank_of, C, M, failed = oracle.filler_pack(price, mem, load0, [0.0] * n_ranks, F, 1.0)
    assert failed is None
    assert rank_of == _lpt(price, load0)
    assert sum(C) == sum(price) + sum(load0)
    assert M == [0.0] * n_ranks


@pytest.mark.parametrize("seed", range(20))
def test_graham_lpt_bound_against_brute_force(seed):
    """From empty ranks, LPT's makespan is at most (4/3 - 1/(3N)) times the
    optimum (Graham 1969); the optimum here is brute force."""
    rng = random.Random(100 + seed)
    n_ranks = rng.randint(2, 3)
    n = rng.randint(n_ranks + 1, 7)
    price = [float(rng.randint(1, 20)) for _ in range(n)]
    F = oracle.load_floor(price, n_ranks)
    rank_of, C, _, failed = oracle.filler_pack(price, [[0.0] * n_ranks] * n, [0.0] * n_ranks, [0.0] * n_ranks, F,
                                               1.0)
    assert failed is None
    opt = min(max(sum(p for p, r in zip(price, a) if r == k) for k in range(n_ranks))
              for a in itertools.product(range(n_ranks), repeat=n))
    assert max(C) <= (4.0 / 3.0 - 1.0 / (3 * n_ranks)) * opt + 1e-12


@pytest.mark.parametrize("seed", range(12))
def test_reduces_to_worst_fit_when_compute_is_free(seed):
    """Zero-price fillers on equally loaded ranks: rho^C = 1 >= rho^M, so
    Eq. 8 maximises the memory slack: worst fit in input order, failing on
    the same item."""
    rng = random.Random(200 + seed)
    n_ranks = rng.randint(2, 6)
    n = rng.randint(1, 30)
    cap = 100.0
    used0 = [float(rng.randint(0, 60)) for _ in range(n_ranks)]
    need = [float(rng.randint(0, 25)) for _ in range(n)]
    mem = [[x] * n_ranks for x in need]
    rank_of, C, M, failed = oracle.filler_pack([0.0] * n, mem, [0.0] * n_ranks, used0, 7.0, cap)
    ref, ref_failed = _worst_fit(need, [cap - u for u in used0])
    assert failed == ref_failed
    assert rank_of[:len(ref)] == ref
    assert all(m <= cap for m in M)


def test_memory_decides_when_it_is_tighter():
    # F = 10, M_cap = 10; C = [0, 4], M = [8, 0]; filler p = 2, M_s = 1 on both ranks.
    # rank 0: rho^C = (10 - 0 - 2)/10 = 0.8, rho^M = (10 - 8 - 1)/10 = 0.1 -> 0.1
    # rank 1: rho^C = (10 - 4 - 2)/10 = 0.4, rho^M = (10 - 0 - 1)/10 = 0.9 -> 0.4
    # rank 1 wins although rank 0 has more compute headroom.
    rank_of, C, M, failed = oracle.filler_pack([2.0], [[1.0, 1.0]], [0.0, 4.0], [8.0, 0.0], 10.0, 10.0)
    assert (rank_of, C, M, failed) == ([1], [0.0, 6.0], [8.0, 1.0], None)


def test_compute_decides_when_it_is_tighter():
    # C = [0, 9], M = [2, 0]; filler p = 2, M_s = 1.
    # rank 0: rho^C = 0.8, rho^M = (10 - 2 - 1)/10 = 0.7 -> 0.7
    # rank 1: rho^C = (10 - 9 - 2)/10 = -0.1               -> -0.1
    rank_of, C, M, failed = oracle.filler_pack([2.0], [[1.0, 1.0]], [0.0, 9.0], [2.0, 0.0], 10.0, 10.0)
    assert (rank_of, C, M, failed) == ([0], [2.0, 9.0], [3.0, 0.0], None)


def test_rank_dependent_memory_and_infeasible_ranks():
    # the filler fits only on rank 2 (its memory there is smaller), whatever the compute slack
    rank_of, _, M, failed = oracle.filler_pack([5.0], [[4.0, 4.0, 1.0]], [0.0, 0.0, 9.0], [7.0, 7.0, 8.0], 10.0,
                                               10.0)
    assert rank_of == [2] and M == [7.0, 7.0, 9.0] and failed is None
    # fits nowhere: planning fails on it, nothing is placed
    rank_of, C, M, failed = oracle.filler_pack([5.0, 1.0], [[4.0, 4.0, 3.0], [0.0] * 3], [0.0] * 3, [7.0, 7.0, 8.0],
                                               10.0, 10.0)
    assert failed == 0 and rank_of == [-1, -1] and C == [0.0] * 3


def test_order_is_decreasing_price():
    # two ranks, equal anchors: the 7 is placed first (rank 0), then 5 (rank 1), then 3 (rank 1)
    rank_of, C, _, _ = oracle.filler_pack([3.0, 7.0, 5.0], [[0.0, 0.0]] * 3, [0.0, 0.0], [0.0, 0.0], 7.5, 1.0)
    assert rank_of == [1, 0, 1] and C == [7.0, 8.0]


@pytest.mark.parametrize("seed", range(8))
def test_scale_invariance(seed):
    """rho^C and rho^M are normalised by F and M_cap, so scaling all times
    (prices, loads, F) or all memory (M_s, M_r, M_cap) by a power of two, which
    is exact, changes no decision."""
    rng = random.Random(300 + seed)
    n_ranks, n = rng.randint(2, 6), rng.randint(1, 30)
    price = [rng.uniform(0.1, 10.0) for _ in range(n)]
    load0 = [rng.uniform(0.0, 20.0) for _ in range(n_ranks)]
    mem = [[rng.uniform(0.0, 10.0) for _ in range(n_ranks)] for _ in range(n)]
    used0 = [rng.uniform(0.0, 40.0) for _ in range(n_ranks)]
    F = oracle.load_floor(price + load0, n_ranks)
    cap = 100.0
    base = oracle.filler_pack(price, mem, load0, used0, F, cap)
    t, m = 2.0 ** rng.randint(-20, 20), 2.0 ** rng.randint(-20, 20)
    scaled = oracle.filler_pack([p * t for p in price], [[x * m for x in row] for row in mem], [c * t for c in load0],
                                [u * m for u in used0], F * t, cap * m)
    assert scaled[0] == base[0] and scaled[3] == base[3]


@pytest.mark.parametrize("seed", range(10))
def test_ledgers_and_memory_feasibility(seed):
    rng = random.Random(400 + seed)
    n_ranks, n = rng.randint(1, 8), rng.randint(1, 60)
    price = [rng.uniform(0.0, 5.0) for _ in range(n)]
    mem = [[rng.uniform(0.0, 3.0) for _ in range(n_ranks)] for _ in range(n)]
    load0 = [rng.uniform(0.0, 30.0) for _ in range(n_ranks)]
    used0 = [rng.uniform(0.0, 20.0) for _ in range(n_ranks)]
    cap = 30.0
    rank_of, C, M, failed = oracle.filler_pack(price, mem, load0, used0, oracle.load_floor(price + load0, n_ranks),
                                               cap)
    placed = [s for s in range(n) if rank_of[s] >= 0]
    for r in range(n_ranks):
        assert C[r] == pytest.approx(load0[r] + sum(price[s] for s in placed if rank_of[s] == r), abs=1e-9)
        assert M[r] == pytest.approx(used0[r] + sum(mem[s][r] for s in placed if rank_of[s] == r), abs=1e-9)
        assert M[r] <= cap
    if failed is not None:
        # every filler more expensive than the failing one was placed; the failing one fits nowhere
        assert all(rank_of[s] >= 0 for s in range(n) if price[s] > price[failed])
        assert all(cap - M[r] < mem[failed][r] for r in range(n_ranks))


def test_rejects_nonpositive_normalisers():
    with pytest.raises(ValueError):
        oracle.filler_pack([1.0], [[0.0]], [0.0], [0.0], 0.0, 1.0)
    with pytest.raises(ValueError):
        oracle.filler_pack([1.0], [[0.0]], [0.0], [0.0], 1.0, 0.0)


def test_compute_slack_counts_the_fillers_own_price():
    # F = 10, M_cap = 10; C = [0, 3], M = [5, 0]; filler p = 6, M_s = 0.
    # rank 0: rho^C = (10 - 0 - 6)/10 = 0.4, rho^M = 0.5 -> 0.4
    # rank 1: rho^C = (10 - 3 - 6)/10 = 0.1, rho^M = 1.0 -> 0.1
    # rank 0 wins; without the -p_s term the minimum would switch to memory on rank 0 (0.5 < 0.7).
    rank_of, _, _, _ = oracle.filler_pack([6.0], [[0.0, 0.0]], [0.0, 3.0], [5.0, 0.0], 10.0, 10.0)
    assert rank_of == [0]


def test_exact_fit_is_feasible():
    # headroom 10 - 6 = 4 holds a filler of exactly 4 (R_s uses >=)
    rank_of, _, M, failed = oracle.filler_pack([1.0], [[4.0]], [0.0], [6.0], 1.0, 10.0)
    assert rank_of == [0] and M == [10.0] and failed is None
