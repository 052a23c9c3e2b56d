"""Routing of a packed whole+shard batch, derived independently of the library.

TEST INFRASTRUCTURE (see the package docstring).

Sec. IV-D of the paper lowers a placement into a rank-local schedule: each
rank materialises only its assigned tokens from the sequences' global token
ranges, sorts its segments deterministically (by split degree, largest
first, with the global placement settling ties) and runs every whole
sequence in one block-diagonal call.  Here a "segment" is what one rank holds of one sequence: a whole
sequence, configuration (1,1,1) in Sec. IV-A, or a local query shard that
attends to a list of K/V blocks (the ring axis of Tab. II).

``row_routing`` states, for every packed query row, where its result goes.
``work_items`` states the canonical list of work items one launch must cover
and the order the scheduler must emit them in:
  * forward: one item per (segment, head, query tile of ``block_m`` rows,
    K/V range of the segment);
  * backward: one item per (segment, head, K/V range, key tile of
    ``block_n`` keys), each item covering all of the segment's query rows
    (none, for a shard without query rows: its keys' gradient is zero).
Cost of an item = rows x keys (attention work is quadratic, Sec. II-A).  The
order is cost descending, ties broken by (segment, head, q_start, k_start,
range index) ascending: the Sec. IV-D segment ordering (largest first, a
fixed input order settling ties) carried over to work items.

An item is the 8-tuple
  (q_start, q_len, k_start, k_len, head, slot, segment, range)
with slot = the CP block index of the range for a shard, -1 for a whole
segment.
"""
from __future__ import annotations

WHOLE = 0
SHARD = 1


def _f(desc, name):
    if isinstance(desc, dict):
        return desc[name]
    return getattr(desc, name)


def row_routing(desc):
    """Per packed query row: (segment, kind, global position, slots).

    ``slots`` is the tuple of partial slots the row is written to (empty for
    a whole row, whose final output goes straight to ``out``).
    """
    cq = _f(desc, "cu_seqlens_q")
    kinds = _f(desc, "kind")
    qoff = _f(desc, "q_offset")
    first = _f(desc, "kv_first")
    count = _f(desc, "kv_count")
    bidx = _f(desc, "block_index")
    rows = []
    for s in range(len(kinds)):
        slots = ()
        if int(kinds[s]) == SHARD:
            slots = tuple(int(bidx[j]) for j in range(int(first[s]), int(first[s]) + int(count[s])))
        for r in range(int(cq[s]), int(cq[s + 1])):
            rows.append((s, int(kinds[s]), int(qoff[s]) + (r - int(cq[s])), slots))
    return rows


def work_items(desc, num_heads, op, block_m, block_n):
    """Canonical, ordered work-item list of one launch.

    op 0: forward; op 1: backward key tiles (dK, dV); op 2: backward query
    tiles that cover every key of the segment, all of its ranges (dQ).
    """
    cq = _f(desc, "cu_seqlens_q")
    ck = _f(desc, "cu_seqlens_k")
    kinds = _f(desc, "kind")
    first = _f(desc, "kv_first")
    count = _f(desc, "kv_count")
    bidx = _f(desc, "block_index")
    items = []
    for s in range(len(kinds)):
        q0, q1 = int(cq[s]), int(cq[s + 1])
        lq = q1 - q0
        # A segment without query rows has no forward or dQ work; its ranges
        # still get key-tile items, since their dK/dV (zero: no query attends
        # to them) is part of the backward's output.
        if lq == 0 and op != 1:
            continue
        shard = int(kinds[s]) == SHARD
        if op == 2:
            j0 = int(first[s])
            j1 = j0 + int(count[s])
            total = sum(int(ck[j + 1]) - int(ck[j]) for j in range(j0, j1))
            for h in range(num_heads):
                for t0 in range(q0, q1, block_m):
                    items.append((t0, min(block_m, q1 - t0), int(ck[j0]), total, h, -1, s, j0))
            continue
        for j in range(int(first[s]), int(first[s]) + int(count[s])):
            k0, k1 = int(ck[j]), int(ck[j + 1])
            lk = k1 - k0
            slot = int(bidx[j]) if shard else -1
            for h in range(num_heads):
                if op == 0:
                    for t0 in range(q0, q1, block_m):
                        tl = min(block_m, q1 - t0)
                        items.append((t0, tl, k0, lk, h, slot, s, j))
                else:
                    for t0 in range(k0, k1, block_n):
                        tl = min(block_n, k1 - t0)
                        items.append((q0, lq, t0, tl, h, slot, s, j))
    items.sort(key=lambda it: (-(it[1] * it[3]), it[6], it[4], it[0], it[2], it[7]))
    return items
