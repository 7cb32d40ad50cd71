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

This oracle rescans a bitmap on every call (O(P)); it is slow on purpose.

Parity: the policy itself is underspecified in the paper, so agreement with
the paper's allocator is "parity unpinned".  The reading above is pinned in
``tests/test_oracle_alloc.py`` by exhaustive minimal-segment optimality over
every free bitmap of small pools, best-fit and head placement checked against
brute-force enumeration, conservation and no-double-assignment invariants, and
the published SplitMix64 output for seed 0.
"""

from __future__ import annotations

from collections import deque
from typing import List, Sequence

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


def free_runs_of(used: Sequence[int]) -> List[tuple]:
    """Maximal runs ``(start, length)`` of zero entries, ascending by start."""
    runs = []
    i, P = 0, len(used)
    while i < P:
        if used[i]:
            i += 1
            continue
        j = i
        while j < P and not used[j]:
            j += 1
        runs.append((i, j - i))
        i = j
    return runs


class RefAllocator:
    def __init__(self, num_blocks: int, policy: int = POLICY_SEGMENT, seed: int = 0):
        if num_blocks < 0:
            raise AllocError("inval", "negative pool size")
        if policy not in (POLICY_SEGMENT, POLICY_FIFO_SORTED, POLICY_FIFO_SHUFFLED):
            raise AllocError("inval", f"unknown policy {policy}")
        self.num_blocks = num_blocks
        self.policy = policy
        self.used = bytearray(num_blocks)
        if policy == POLICY_FIFO_SORTED:
            self.fifo = deque(range(num_blocks))
        elif policy == POLICY_FIFO_SHUFFLED:
            self.fifo = deque(shuffled_ids(num_blocks, seed))
        else:
            self.fifo = None

    # -- queries -----------------------------------------------------------
    def free_count(self) -> int:
        return self.num_blocks - sum(self.used)

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
            runs = free_runs_of(self.used)
            need = n
            while need > 0:
                fitting = [r for r in runs if r[1] >= need]
                if fitting:
                    start, _ = min(fitting, key=lambda r: (r[1], r[0]))
                    out.extend(range(start, start + need))
                    need = 0
                else:
                    big = max(runs, key=lambda r: (r[1], -r[0]))
                    runs.remove(big)
                    out.extend(range(big[0], big[0] + big[1]))
                    need -= big[1]
        for b in out:
            self.used[b] = 1
        return out

    def _validate(self, ids: Sequence[int], want_used: bool):
        seen = set()
        for b in ids:
            b = int(b)
            if b < 0 or b >= self.num_blocks:
                raise AllocError("range", f"block {b} outside [0, {self.num_blocks})")
            if b in seen:
                raise AllocError("dup", f"block {b} listed twice")
            seen.add(b)
        for b in ids:
            if bool(self.used[int(b)]) != want_used:
                raise AllocError("dup", f"block {int(b)} is {'free' if want_used else 'in use'}")

    def free(self, ids: Sequence[int]) -> None:
        self._validate(ids, want_used=True)
        for b in ids:
            self.used[int(b)] = 0
        if self.fifo is not None:
            self.fifo.extend(int(b) for b in ids)

    def mark_used(self, ids: Sequence[int]) -> None:
        self._validate(ids, want_used=False)
        for b in ids:
            self.used[int(b)] = 1
        if self.fifo is not None:
            gone = set(int(b) for b in ids)
            self.fifo = deque(b for b in self.fifo if b not in gone)
