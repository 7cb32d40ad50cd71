"""CPU oracle for the FlowKV KV-cache transfer path (arXiv 2504.03775).

TEST INFRASTRUCTURE ONLY.  Nothing in the product package imports, calls or
links anything here; only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may use it.  It shares no code, header,
table or helper with the HIP path.

What it computes, each piece written from the paper's description:

* :mod:`oracle.kvcopy`  -- the transfer result itself: every token slot of a
  request's K and V, in every layer, lands in the receiver's block that the
  receiver's block list names for it.  The two pool layouts are the two sides
  of Eq. 5 (section 3.3): per-layer tensors ``(L, 2, B, H)`` and the
  restructured block-major tensor ``(B, L, 2, H)``.
* :mod:`oracle.plan`    -- bidirectional segment alignment (section 3.3 and the
  Figure 3 caption): the maximal runs of logical positions whose block IDs
  advance by one in lockstep on the sending and the receiving side.
* :mod:`oracle.alloc`   -- the segment-based, contiguity-aware block allocator
  of section 3.3 (best-fit over free segments, merge on free), plus the two
  naive free-list policies used to build fragmented tables.
* :mod:`oracle.attention` -- decode attention over a paged pool in either
  layout (the PagedAttention consumer section 3.3 adapts), float64.
* :mod:`oracle.scheduler` -- the Load-Aware Scheduler's evaluation and
  routing (section 3.4, Algorithm 1), float64, term by term.

Parity status of each function is stated in its module header.
"""

from .kvcopy import (  # noqa: F401
    LAYER_MAJOR,
    BLOCK_MAJOR,
    HostPool,
    slot_address,
    transfer_ref,
    transfer_fast,
    transfer_batch_fast,
)
from .plan import plan_ref, plan_batch_ref  # noqa: F401
from .alloc import (  # noqa: F401
    RefAllocator,
    NoSpace,
    AllocError,
    POLICY_SEGMENT,
    POLICY_FIFO_SORTED,
    POLICY_FIFO_SHUFFLED,
    splitmix64_stream,
    shuffled_ids,
)
