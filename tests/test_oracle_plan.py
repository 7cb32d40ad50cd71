"""Pins for the segment-alignment oracle (``oracle.plan``), CPU only.

The oracle scans for breaks.  These tests pin it by exhaustive search over
every way to cut a request's block lists into lockstep-contiguous pieces (the
fewest pieces is the alignment; it is unique), by hand-worked cases from the
paper's description, and by the contiguous and stride-2 special cases.
"""

import itertools
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import plan_batch_ref, plan_ref

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "plan_cases.json")


def piece_ok(S, D):
    return all(S[j] == S[0] + j and D[j] == D[0] + j for j in range(len(S)))


def brute_force_plan(S, D):
    """Fewest pieces over all 2^(n-1) cut sets; returns the pieces."""
    n = len(S)
    if n == 0:
        return []
    best = None
    for mask in range(1 << (n - 1)):
        cuts = [0] + [i + 1 for i in range(n - 1) if mask >> i & 1] + [n]
        pieces = list(zip(cuts[:-1], cuts[1:]))
        if all(piece_ok(S[a:b], D[a:b]) for a, b in pieces):
            if best is None or len(pieces) < len(best):
                best = pieces
            elif len(pieces) == len(best):
                assert pieces == best, "fewest-piece cut must be unique"
    return [(S[a], D[a], b - a) for a, b in best]


def test_exhaustive_small_lists():
    pool = range(5)
    count = 0
    for n in range(0, 4):
        for S in itertools.permutations(pool, n):
            for D in itertools.permutations(pool, n):
                assert plan_ref(S, D) == brute_force_plan(S, D), (S, D)
                count += 1
    assert count == 1 + 25 + 400 + 3600


@settings(max_examples=300, deadline=None)
@given(st.data())
def test_random_lists_match_brute_force(data):
    n = data.draw(st.integers(0, 9))
    # draw from a small space so contiguous runs are common
    S = data.draw(st.lists(st.integers(0, 12), min_size=n, max_size=n, unique=True))
    D = data.draw(st.lists(st.integers(0, 12), min_size=n, max_size=n, unique=True))
    assert plan_ref(S, D) == brute_force_plan(S, D)


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["name"])
def test_golden_cases(case):
    got = [list(s) for s in plan_ref(case["S"], case["D"])]
    assert got == case["segments"]


def test_special_cases():
    n = 813
    assert plan_ref(list(range(100, 100 + n)), list(range(7, 7 + n))) == [(100, 7, n)]
    S = [2 * i for i in range(n)]
    D = [2 * i + 1 for i in range(n)]
    assert len(plan_ref(S, D)) == n


@settings(max_examples=200, deadline=None)
@given(st.data())
def test_segments_reassemble_lists_and_are_maximal(data):
    n = data.draw(st.integers(0, 64))
    seed = data.draw(st.integers(0, 2**32 - 1))
    rng = np.random.default_rng(seed)
    # runs of random length from a shuffled set of run starts
    S = list(rng.permutation(200)[:n])
    D = list(rng.permutation(200)[:n])
    # make some stretches contiguous on both sides
    for i in range(1, n):
        if rng.random() < 0.6:
            S[i], D[i] = S[i - 1] + 1, D[i - 1] + 1
    if len(set(S)) < n or len(set(D)) < n:
        return
    segs = plan_ref(S, D)
    rs, rd = [], []
    for s, d, m in segs:
        rs.extend(range(s, s + m))
        rd.extend(range(d, d + m))
    assert rs == list(S) and rd == list(D)
    pos = 0
    for k, (s, d, m) in enumerate(segs):
        if k > 0:  # not mergeable with the previous segment
            ps, pd, pm = segs[k - 1]
            assert not (s == ps + pm and d == pd + pm)
        pos += m


def test_batch_never_crosses_requests():
    tables = [([0, 1, 2], [10, 11, 12]), ([3, 4], [13, 14])]
    # the two requests would form one run if concatenated
    assert plan_batch_ref(tables) == [(0, 10, 3, 0), (3, 13, 2, 1)]
    assert plan_batch_ref([]) == []
