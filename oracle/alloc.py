"""Oracle for the contiguity-aware block allocator (test infrastructure only).

Section 3.3 of FlowKV (arXiv 2504.03775) describes the allocator in one
paragraph: free blocks are managed as segments (kept in minimum heaps), a new
request is placed in one or a few contiguous segments, the segments chosen are
the ones that waste least, and adjacent free segments are merged on release.
The paper gives no further rule, so this oracle takes the following reading,
step by step:

1. State: which blocks are free.  The free segments are the maximal runs of
   free block IDs; merging adjacent free segments on release is automatic
   because the runs are recomputed from the free set on every call.
2. ``alloc(n)``: fail (state unchanged) when fewer than ``n`` blocks are free.
   If some free run holds at least ``n`` blocks, take the best fit -- the
   shortest such run, the lowest start on ties -- and hand out its first ``n``
   blocks in ascending order.  Otherwise take the longest run whole (lowest
   start on ties), append its blocks in ascending order, and repeat with the
   remainder until the remainder fits one run, which is then best-fitted.
   The returned list is in the order taken (the request's logical order).
3. ``free(ids)``: all IDs must be in range, distinct and in use; they become
   free.  ``mark_used(ids)``: all in range, distinct and free; they become used
   (a decode node's resident requests).

Two naive free-list policies build the fragmented tables the paper contrasts
with: a FIFO of free IDs that starts ascending (``POLICY_FIFO_SORTED``) or
starts as a seeded Fisher-Yates shuffle (``POLICY_FIFO_SHUFFLED``); ``alloc``
pops from the front, ``free`` appends in table order, ``mark_used`` removes.
The shuffle draws from SplitMix64 (Steele, Lea and Flood, "Fast splittable
pseudorandom number generators", OOPSLA 2014): for ``i`` from ``P-1`` down to
1, swap slot ``i`` with slot ``next() mod (i+1)``, the state starting at the
seed.

This oracle rescans the free flags on every call (O(P)); it is slow on purpose.

Parity: the policy itself is underspecified in the paper, so agreement with
the paper's allocator is "parity unpinned".  The reading above is pinned in
``tests/test_oracle_alloc.py`` by exhaustive minimal-segment optimality over
every free bitmap of small pools, best-fit and head placement checked against
brute-force enumeration, conservation and no-double-assignment invariants,
the published SplitMix64 output for seed 0, and the shuffle reaching every
order of 3 and 4 blocks about equally often over consecutive seeds.
"""

from __future__ import annotations

from collections import deque
from typing import List, Sequence

import numpy as np

POLICY_SEGMENT = 0
POLICY_FIFO_SORTED = 1
POLICY_FIFO_SHUFFLED = 2

_MASK64 = (1 << 64) - 1


class AllocError(Exception):
    """Rejected call; ``kind`` is one of 'range', 'dup', 'nospace', 'inval'."""

    def __init__(self, kind: str, msg: str):
        super().__init__(msg)
        self.kind = kind


class NoSpace(AllocError):
    def __init__(self, msg: str):
        super().__init__("nospace", msg)


def splitmix64_stream(seed: int):
    """Yield SplitMix64 outputs for the given 64-bit seed."""
    state = seed & _MASK64
    while True:
        state = (state + 0x9E3779B97F4A7C15) & _MASK64
        z = state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
        yield z ^ (z >> 31)


def shuffled_ids(num_blocks: int, seed: int) -> List[int]:
    a = list(range(num_blocks))
    rng = splitmix64_stream(seed)
    for i in range(num_blocks - 1, 0, -1):
        j = next(rng) % (i + 1)
        a[i], a[j] = a[j], a[i]
    return a


def free_run_arrays(used):
    """Starts and lengths of the maximal runs of zero entries, ascending by
    start.  A run starts where the used-flag falls from 1 to 0 (or at the
    start) and ends where it rises again (or at the end)."""
    u = np.asarray(used, dtype=np.int8)
    edges = np.diff(np.concatenate(([1], u, [1])))
    starts = np.flatnonzero(edges == -1)
    ends = np.flatnonzero(edges == 1)
    return starts, ends - starts


def free_runs_of(used) -> List[tuple]:
    """Maximal free runs as ``(start, length)`` tuples, ascending by start."""
    starts, lens = free_run_arrays(used)
    return [(int(a), int(b)) for a, b in zip(starts, lens)]


class RefAllocator:
    def __init__(self, num_blocks: int, policy: int = POLICY_SEGMENT, seed: int = 0):
        if num_blocks < 0:
            raise AllocError("inval", "negative pool size")
        if policy not in (POLICY_SEGMENT, POLICY_FIFO_SORTED, POLICY_FIFO_SHUFFLED):
            raise AllocError("inval", f"unknown policy {policy}")
        self.num_blocks = num_blocks
        self.policy = policy
        self.used = np.zeros(num_blocks, dtype=np.uint8)
        if policy == POLICY_FIFO_SORTED:
            self.fifo = deque(range(num_blocks))
        elif policy == POLICY_FIFO_SHUFFLED:
            self.fifo = deque(shuffled_ids(num_blocks, seed))
        else:
            self.fifo = None

    # -- queries -----------------------------------------------------------
    def free_count(self) -> int:
        return self.num_blocks - int(self.used.sum())

    def stats(self):
        runs = free_runs_of(self.used)
        return {
            "free_blocks": self.free_count(),
            "free_segments": len(runs),
            "largest_free": max((r[1] for r in runs), default=0),
        }

    # -- operations --------------------------------------------------------
    def alloc(self, n: int) -> List[int]:
        if n < 0:
            raise AllocError("inval", "negative block count")
        if n > self.free_count():
            raise NoSpace(f"{n} blocks asked, {self.free_count()} free")
        if self.policy != POLICY_SEGMENT:
            out = [self.fifo.popleft() for _ in range(n)]
        else:
            out = []
            starts, lens = free_run_arrays(self.used)
            need = n
            while need > 0:
                fitting = np.flatnonzero(lens >= need)
                if fitting.size:
                    # shortest fitting run; argmin keeps the first (lowest
                    # start) of equally short runs
                    k = fitting[np.argmin(lens[fitting])]
                    out.extend(range(int(starts[k]), int(starts[k]) + need))
                    need = 0
                else:
                    # longest run, taken whole; argmax keeps the lowest start
                    k = int(np.argmax(lens))
                    out.extend(range(int(starts[k]), int(starts[k] + lens[k])))
                    need -= int(lens[k])
                    starts, lens = np.delete(starts, k), np.delete(lens, k)
        self.used[np.asarray(out, dtype=np.int64)] = 1
        return out

    def _validate(self, ids: Sequence[int], want_used: bool) -> np.ndarray:
        a = np.asarray(ids, dtype=np.int64).reshape(-1)
        bad = a[(a < 0) | (a >= self.num_blocks)]
        if bad.size:
            raise AllocError("range", f"block {int(bad[0])} outside [0, {self.num_blocks})")
        if np.unique(a).size != a.size:
            raise AllocError("dup", "a block is listed twice")
        wrong = a[self.used[a].astype(bool) != want_used]
        if wrong.size:
            raise AllocError("dup", f"block {int(wrong[0])} is {'free' if want_used else 'in use'}")
        return a

    def free(self, ids: Sequence[int]) -> None:
        a = self._validate(ids, want_used=True)
        self.used[a] = 0
        if self.fifo is not None:
            self.fifo.extend(int(b) for b in a)

    def mark_used(self, ids: Sequence[int]) -> None:
        a = self._validate(ids, want_used=False)
        self.used[a] = 1
        if self.fifo is not None:
            gone = set(int(b) for b in a)
            self.fifo = deque(b for b in self.fifo if b not in gone)
