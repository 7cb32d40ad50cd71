"""Pins for the allocator oracle (``oracle.alloc``), CPU only.

The paper's allocator policy is one paragraph (section 3.3); agreement with
the paper's own code is "parity unpinned".  What is pinned here is the
reading the oracle states: fewest segments possible for every request, best
fit with head placement when one segment suffices, never a block handed out
twice, failure leaves the state unchanged, and the naive policies' free-list
order including the published SplitMix64 output.
"""

import itertools

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import (POLICY_FIFO_SHUFFLED, POLICY_FIFO_SORTED, POLICY_SEGMENT,
                    AllocError, NoSpace, RefAllocator, shuffled_ids,
                    splitmix64_stream)


def runs_in_order(ids):
    """Number of ascending +1 runs in a list, in its own order."""
    return sum(1 for i in range(len(ids)) if i == 0 or ids[i] != ids[i - 1] + 1)


def free_runs_groupby(bits):
    """(start, length) of maximal free runs, via itertools.groupby."""
    out, pos = [], 0
    for used, grp in itertools.groupby(bits):
        k = len(list(grp))
        if not used:
            out.append((pos, k))
        pos += k
    return out


def fewest_runs_needed(runs, n):
    lens = sorted((r[1] for r in runs), reverse=True)
    tot = 0
    for k, v in enumerate(lens, 1):
        tot += v
        if tot >= n:
            return k
    return None


def test_minimal_segments_every_bitmap():
    """P = 11: every free bitmap and every feasible n."""
    P = 11
    cases = 0
    for mask in range(1 << P):
        bits = [(mask >> i) & 1 for i in range(P)]
        runs = free_runs_groupby(bits)
        nfree = P - sum(bits)
        for n in range(1, nfree + 1):
            a = RefAllocator(P, POLICY_SEGMENT)
            a.mark_used([i for i in range(P) if bits[i]])
            ids = a.alloc(n)
            assert len(ids) == n and len(set(ids)) == n
            assert all(not bits[i] for i in ids)
            assert runs_in_order(ids) == fewest_runs_needed(runs, n), (bits, n, ids)
            cases += 1
    assert cases == sum(P - bin(m).count("1") for m in range(1 << P))


def test_best_fit_head_placement_every_bitmap():
    P = 10
    for mask in range(1 << P):
        bits = [(mask >> i) & 1 for i in range(P)]
        runs = free_runs_groupby(bits)
        for n in range(1, max((r[1] for r in runs), default=0) + 1):
            fitting = [r for r in runs if r[1] >= n]
            start = min(fitting, key=lambda r: (r[1], r[0]))[0]
            a = RefAllocator(P, POLICY_SEGMENT)
            a.mark_used([i for i in range(P) if bits[i]])
            assert a.alloc(n) == list(range(start, start + n))


def test_multi_segment_takes_largest_runs_whole():
    # free runs: [0,2) len 2, [3,7) len 4, [8,11) len 3, [12,13) len 1
    bits = [0, 0, 1, 0, 0, 0, 0, 1, 0, 0, 0, 1, 0]
    a = RefAllocator(len(bits), POLICY_SEGMENT)
    a.mark_used([i for i, b in enumerate(bits) if b])
    # 6 blocks: longest run (4) whole, then best fit for 2 -> the run of 2
    assert a.alloc(6) == [3, 4, 5, 6, 0, 1]
    # remaining runs: [8,11) len 3, [12,13) len 1; 4 blocks -> 3 whole + 1
    assert a.alloc(4) == [8, 9, 10, 12]


def test_free_merges_neighbours():
    a = RefAllocator(8, POLICY_SEGMENT)
    x = a.alloc(3)
    y = a.alloc(2)
    z = a.alloc(3)
    assert (x, y, z) == ([0, 1, 2], [3, 4], [5, 6, 7])
    a.free(x)
    a.free(z)
    assert a.stats() == {"free_blocks": 6, "free_segments": 2, "largest_free": 3}
    a.free(y)
    assert a.stats() == {"free_blocks": 8, "free_segments": 1, "largest_free": 8}
    assert a.alloc(8) == list(range(8))


def test_errors_leave_state_unchanged():
    a = RefAllocator(6, POLICY_SEGMENT)
    got = a.alloc(4)
    before = (a.used.tobytes(), a.stats())
    with pytest.raises(NoSpace):
        a.alloc(3)
    for bad, kind in (([9], "range"), ([-1], "range"), ([0, 0], "dup"), ([4], "dup")):
        with pytest.raises(AllocError) as e:
            a.free(bad)
        assert e.value.kind == kind
    with pytest.raises(AllocError):
        a.mark_used([got[0]])
    with pytest.raises(AllocError):
        a.alloc(-1)
    assert (a.used.tobytes(), a.stats()) == before
    assert a.alloc(0) == []


@pytest.mark.parametrize("policy", [POLICY_SEGMENT, POLICY_FIFO_SORTED, POLICY_FIFO_SHUFFLED])
@settings(max_examples=60, deadline=None)
@given(seed=st.integers(0, 2**32 - 1))
def test_random_op_streams_keep_invariants(policy, seed):
    rng = np.random.default_rng(seed)
    P = int(rng.integers(1, 80))
    a = RefAllocator(P, policy, seed=seed)
    pre = [int(x) for x in rng.permutation(P)[: int(rng.integers(0, P // 3 + 1))]]
    a.mark_used(pre)
    live = {}
    for step in range(60):
        if live and rng.random() < 0.45:
            k = list(live)[int(rng.integers(len(live)))]
            a.free(live.pop(k))
        else:
            n = int(rng.integers(0, P // 2 + 2))
            nfree = a.free_count()
            if n > nfree:
                with pytest.raises(NoSpace):
                    a.alloc(n)
                continue
            ids = a.alloc(n)
            live[step] = ids
        handed = [b for ids in live.values() for b in ids] + pre
        assert len(handed) == len(set(handed)), "block handed out twice"
        assert a.free_count() + len(handed) == P
        assert all(a.used[b] for b in handed)


def test_splitmix64_published_output():
    # SplitMix64 (Steele, Lea, Flood 2014) seeded with 0: published first output
    assert next(splitmix64_stream(0)) == 0xE220A8397B1DCDAF


def test_shuffle_is_seeded_fisher_yates():
    P = 3
    # i = 2: swap a[2] with a[r0 % 3]; i = 1: swap a[1] with a[r1 % 2]
    g = splitmix64_stream(5)
    r0, r1 = next(g), next(g)
    a = [0, 1, 2]
    j = r0 % 3
    a[2], a[j] = a[j], a[2]
    j = r1 % 2
    a[1], a[j] = a[j], a[1]
    assert shuffled_ids(P, 5) == a
    big = shuffled_ids(1000, 123)
    assert sorted(big) == list(range(1000)) and big != list(range(1000))
    assert shuffled_ids(1000, 123) == big and shuffled_ids(1000, 124) != big


@pytest.mark.parametrize("P,seeds,chi2_limit", [(3, 6000, 20.5), (4, 24000, 49.7)])
def test_shuffle_reaches_every_permutation_evenly(P, seeds, chi2_limit):
    """Over consecutive seeds the shuffled free list takes each of the P!
    orders about equally often (chi-square under its 0.1% critical value for
    P! - 1 degrees of freedom).  Sattolo's variant (swap index drawn below i,
    not up to i) reaches only the (P-1)! cyclic orders, and a skewed index
    draw shifts the counts; both fail here."""
    import collections
    import itertools

    perms = list(itertools.permutations(range(P)))
    counts = collections.Counter(tuple(shuffled_ids(P, s)) for s in range(seeds))
    assert set(counts) == set(perms)
    expect = seeds / len(perms)
    chi2 = sum((counts[p] - expect) ** 2 / expect for p in perms)
    assert chi2 < chi2_limit, chi2


def test_fifo_policies_order():
    a = RefAllocator(8, POLICY_FIFO_SORTED)
    a.mark_used([1, 4])
    assert a.alloc(3) == [0, 2, 3]
    a.free([2, 0])
    assert a.alloc(5) == [5, 6, 7, 2, 0]
    b = RefAllocator(8, POLICY_FIFO_SHUFFLED, seed=9)
    assert b.alloc(8) == shuffled_ids(8, 9)
