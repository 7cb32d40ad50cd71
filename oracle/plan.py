"""Oracle for bidirectional segment alignment (test infrastructure only).

Section 3.3 and the Figure 3 caption of FlowKV (arXiv 2504.03775): before the
transfer, the sender's and the receiver's block-ID lists are compared and the
runs of blocks that are contiguous on both sides are found; each such run is
moved by one operation, so the fully contiguous case needs one operation
instead of one per block.

Plain definition written out: the segments of a request with sender list
``S`` and receiver list ``D`` (equal length ``n``) are the maximal runs of
consecutive logical positions ``i .. i+m-1`` with ``S[i+j] == S[i] + j`` and
``D[i+j] == D[i] + j`` for every ``j < m``.  A run starts at position 0 and
wherever either list fails to step by +1.  Each segment is recorded as
``(S[i], D[i], m)``.  The decomposition into maximal runs is unique.

In a batch each request is aligned on its own: runs never cross requests.

Parity: pinned in ``tests/test_oracle_plan.py`` by exhaustive search for the
fewest lockstep-contiguous pieces on small lists, hand-worked cases in
``tests/golden/plan_cases.json``, and the fully contiguous / stride-2 special
cases.
"""

from __future__ import annotations

from typing import List, Sequence, Tuple

Segment = Tuple[int, int, int]  # (sender start block, receiver start block, blocks)


def plan_ref(S: Sequence[int], D: Sequence[int]) -> List[Segment]:
    if len(S) != len(D):
        raise ValueError("sender and receiver block lists differ in length")
    segs: List[Segment] = []
    i = 0
    n = len(S)
    while i < n:
        m = 1
        while i + m < n and S[i + m] == S[i] + m and D[i + m] == D[i] + m:
            m += 1
        segs.append((int(S[i]), int(D[i]), m))
        i += m
    return segs


def plan_batch_ref(tables) -> List[Tuple[int, int, int, int]]:
    """Align each request of ``tables = [(S_r, D_r), ...]`` separately.

    Returns ``(src, dst, blocks, request index)`` in request order."""
    out = []
    for r, (S, D) in enumerate(tables):
        out.extend((s, d, m, r) for (s, d, m) in plan_ref(S, D))
    return out
