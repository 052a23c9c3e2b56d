"""Oracle for packed whole+shard attention: TEST INFRASTRUCTURE, not product code.

Plain, slow, fp64 CPU definitions of everything the GPU path computes, written
from the paper's description of the Coalesced Attention Engine (Sec. IV-D) and
of context parallelism (Sec. II-B, Tab. II), plus the standard definitions of
exact softmax attention that the paper relies on (it cites FlashAttention and
ring attention and never writes the formulas itself).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP path and
imports nothing from the product package: descriptors arrive as plain arrays.

Modules
  attention  forward, LSE merge and backward of exact non-causal attention,
             per segment and over a packed whole+shard batch.
  routing    which packed rows go where (segment, kind, global position,
             partial slot) and the canonical set of query-tile work items.
  planner    Filler Packing (Sec. IV-C, Eq. 8): the greedy that places whole
             fillers into the compute and memory headroom the anchors leave.

Every function is pinned by ``tests/test_oracle_*.py`` against things other
than itself: 50-digit ``decimal`` brute force, closed forms, finite
differences, the invariants the paper's exactness claims imply, and for the
planner the textbook greedy rules it reduces to (LPT, worst fit) and Graham's
LPT bound against brute-force optima.  No
function here is "parity unpinned".
"""
from .attention import (  # noqa: F401
    attend,
    attend_bwd,
    attend_bwd_given,
    lse_merge,
    packed_forward,
    packed_backward,
    segment_rows,
)
from .routing import row_routing, work_items  # noqa: F401
from .planner import filler_pack, load_floor  # noqa: F401
