"""Filler Packing, Stage 2 of the two-stage planner (Sec. IV-C, Eq. 8).

TEST INFRASTRUCTURE (see the package docstring).

After Stage 1 has placed the anchors, every rank r has a compute ledger C_r
(its summed per-rank prices) and a memory ledger M_r.  Fillers stay whole
and are placed one at a time, most expensive first (decreasing profiled
whole-sequence price p_s).  With the zero-communication load floor
F = sum over the whole batch of p_s / N, the compute headroom h^C_r = F - C_r
and the memory headroom h^M_r = M_cap - M_r, filler s may go to any rank
whose memory headroom holds its whole-sequence memory M_{s,whole,r}, and
goes to the feasible rank that maximises the smaller of its two normalised
post-placement slacks

    rho^C = (h^C_r - p_s) / F,      rho^M = (h^M_r - M_{s,whole,r}) / M_cap.

The ledgers of the chosen rank are then updated and the next filler scored
against them.  If some filler has no feasible rank, planning fails.

Readings where the paper is silent: fillers of equal price keep their input
order (a stable sort), a tie in the score goes to the lowest rank index, and
both normalisers must be positive.  Everything is fp64, in the order written
above, so the integer decision (which rank) is reproducible.
"""
from __future__ import annotations


def load_floor(whole_prices, num_ranks: int) -> float:
    """F: every sequence of the batch (anchors and fillers) at its whole
    price, spread evenly over the ranks (Sec. IV-C, Stage 2)."""
    total = 0.0
    for p in whole_prices:
        total += float(p)
    return total / num_ranks


def filler_pack(price, mem, load, mem_used, floor: float, mem_cap: float):
    """Eq. 8 over all fillers.

    price     p_s for each filler s
    mem       mem[s][r] = M_{s,whole,r}
    load      C_r after Stage 1 (not modified)
    mem_used  M_r after Stage 1 (not modified)
    Returns (rank_of, C, M, failed): rank_of[s] is r*(s) (-1 when not
    placed), C and M the final ledgers, failed the index of the first filler
    that fit on no rank (None when every filler was placed).
    """
    if not (floor > 0.0 and mem_cap > 0.0):
        raise ValueError("the load floor and the memory cap must be positive")
    n = len(price)
    num_ranks = len(load)
    C = [float(x) for x in load]
    M = [float(x) for x in mem_used]
    rank_of = [-1] * n
    order = sorted(range(n), key=lambda s: -float(price[s]))      # stable: ties keep input order
    for s in order:
        p = float(price[s])
        best_r, best = -1, None
        for r in range(num_ranks):
            need = float(mem[s][r])
            h_m = mem_cap - M[r]
            if not h_m >= need:                 # r is not in R_s
                continue
            h_c = floor - C[r]
            rho_c = (h_c - p) / floor
            rho_m = (h_m - need) / mem_cap
            score = min(rho_c, rho_m)
            if best is None or score > best:    # strict: a tie keeps the lower rank
                best_r, best = r, score
        if best_r < 0:
            return rank_of, C, M, s
        rank_of[s] = best_r
        C[best_r] += p
        M[best_r] += float(mem[s][best_r])
    return rank_of, C, M, None
