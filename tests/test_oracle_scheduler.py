"""Pins for the Load-Aware Scheduler oracle (``oracle.scheduler``), CPU only.

The paper gives Algorithm 1 but no worked example, so the oracle is pinned by
what the algorithm fixes whatever the unstated constants are:

* one-hot weights: each score term reads the indicator Algorithm 1 names for
  it (a swapped index or role fails here);
* the sliding window: constant inputs pass through, a spike leaves the
  window after exactly `window` further samples, and the mean of a ramp is
  its midpoint;
* C^p and C^d average only their own role's nodes;
* hand-worked scenario boundaries (the comparisons are inclusive, on |C|);
* imbalanced load: the idle set and the role it takes, worked by hand;
* extreme load: the scale request arrives on exactly the scale_after-th
  consecutive evaluation and the count restarts after normal load;
* low load (the reading that gives section 3.4's low-load extreme a branch):
  strict lower thresholds tested before normal load, its own persistence
  count, a scale-down only for roles with more than one node, and offline
  nodes left out of averages, idle sets and routes, worked by hand;
* routing: brute force over every (P, D) pair ordered by (TTFT, index),
  then (latency, index), on random small clusters; closed cases for full
  prefix hits and for no decode node with room.
"""

import itertools
import random

import pytest

from oracle.scheduler import (DECODE, EXTREME, IMBALANCED, LOW_LOAD, NORMAL, OFFLINE, PREFILL,
                              Params, RefScheduler, default_params, route)

ONE = [1.0] * 12


def params(**kw):
    base = dict(window=1, scale=list(ONE), w_prefill=[0.0] * 8, w_decode=[0.0] * 8,
                eps_p_low=1.0, eps_d_low=1.0, eps_p_high=2.0, eps_d_high=2.0,
                idle_threshold=0.25, scale_after=2)
    base.update(kw)
    return Params(**base)


def test_one_hot_weights_read_the_named_indicator():
    prefill_idx = [0, 1, 2, 3, 8, 9, 10, 11]   # L_r^p L_w^p L_sw^p L_se^p T_b KV_u G_u MB_u
    decode_idx = [4, 5, 6, 7, 8, 9, 10, 11]    # L_r^d L_w^d L_sw^d L_se^d T_b KV_u G_u MB_u
    status = [float(2 ** k) for k in range(12)]  # every indicator distinct
    for t in range(8):
        w = [0.0] * 8
        w[t] = 1.0
        s = RefScheduler(params(w_prefill=w, w_decode=w), [PREFILL])
        s.observe([status])
        cp, cd = s.node_scores(0)
        assert cp == status[prefill_idx[t]]
        assert cd == status[decode_idx[t]]


def test_normalisation_divides_by_the_scale():
    scale = [float(k + 1) for k in range(12)]
    w = [0.0] * 8
    w[1] = 1.0                                   # L_w^p
    s = RefScheduler(params(scale=scale, w_prefill=w), [PREFILL])
    s.observe([[6.0] * 12])
    assert s.node_scores(0)[0] == 6.0 / 2.0


def test_sliding_window():
    w = [1.0] + [0.0] * 7                        # C^p = L_r^p
    s = RefScheduler(params(window=4, w_prefill=w), [PREFILL])
    for _ in range(6):
        s.observe([[3.0] + [0.0] * 11])
    assert s.node_scores(0)[0] == 3.0            # constant passes through
    s.observe([[103.0] + [0.0] * 11])            # spike
    assert s.node_scores(0)[0] == (3.0 * 3 + 103.0) / 4
    for k in range(3):
        s.observe([[3.0] + [0.0] * 11])
        assert s.node_scores(0)[0] == (3.0 * 3 + 103.0) / 4   # still inside
    s.observe([[3.0] + [0.0] * 11])
    assert s.node_scores(0)[0] == 3.0            # gone after `window` more samples
    r = RefScheduler(params(window=5, w_prefill=w), [PREFILL])
    for v in range(10):                          # ramp 0..9: the last 5 average to 7
        r.observe([[float(v)] + [0.0] * 11])
    assert r.node_scores(0)[0] == 7.0
    fresh = RefScheduler(params(window=8, w_prefill=w), [PREFILL])
    fresh.observe([[2.0] + [0.0] * 11])
    fresh.observe([[4.0] + [0.0] * 11])
    assert fresh.node_scores(0)[0] == 3.0        # partial window: mean of what exists


def test_role_averages_only_their_own_nodes():
    w = [1.0] + [0.0] * 7
    wd = [0.0] * 4 + [1.0] + [0.0] * 3           # C^d = T_b
    s = RefScheduler(params(w_prefill=w, w_decode=wd), [PREFILL, PREFILL, DECODE])
    s.observe([[0.5] + [0.0] * 11, [0.25] + [0.0] * 11,
               [1000.0] * 8 + [0.75] + [0.0] * 3])  # the decode node's L_r^p is huge
    r = s.evaluate()
    assert r.c_prefill == (0.5 + 0.25) / 2
    assert r.c_decode == 0.75
    s.set_role(2, PREFILL)                       # now it counts for C^p, and C^d has no node
    r = s.evaluate()
    assert r.c_prefill == (0.5 + 0.25 + 1000.0) / 3 and r.c_decode == 0.0


@pytest.mark.parametrize("cp,cd,want", [
    (1.0, 1.0, NORMAL),        # inclusive at the low thresholds
    (-1.0, 0.0, NORMAL),       # |C|
    (1.0000001, 0.0, IMBALANCED),
    (0.0, 2.0, IMBALANCED),    # inclusive at the high thresholds
    (2.0, 2.0, IMBALANCED),
    (2.0000001, 0.0, EXTREME),
    (0.0, -2.5, EXTREME),
])
def test_scenario_boundaries(cp, cd, want):
    w = [1.0] + [0.0] * 7
    wd = [0.0, 0.0, 0.0, 0.0, 1.0, 0.0, 0.0, 0.0]   # C^d = T_b
    s = RefScheduler(params(w_prefill=w, w_decode=wd), [PREFILL, DECODE])
    s.observe([[cp] + [0.0] * 11, [0.0] * 8 + [cd, 0.0, 0.0, 0.0]])
    assert s.evaluate().scenario == want


def test_imbalanced_idle_nodes_worked_by_hand():
    # 2 prefill nodes with C^p 1.5 and 1.25 (mean 1.375: above low 1, under
    # high 2); 3 decode nodes with C^d 0.125, 0.5, 0.0625 (mean 0.229).
    # Prefill is busier (1.375 / 1 >= 0.229 / 1); decode nodes under the
    # 0.25 idle threshold are 2 and 4; they take the prefill role.
    w = [1.0] + [0.0] * 7
    wd = [0.0] * 4 + [1.0] + [0.0] * 3
    s = RefScheduler(params(w_prefill=w, w_decode=wd), [PREFILL, PREFILL, DECODE, DECODE, DECODE])
    st = [[1.5] + [0.0] * 11, [1.25] + [0.0] * 11,
          [0.0] * 8 + [0.125, 0, 0, 0], [0.0] * 8 + [0.5, 0, 0, 0], [0.0] * 8 + [0.0625, 0, 0, 0]]
    s.observe(st)
    r = s.evaluate()
    assert r.scenario == IMBALANCED and r.switch_to == PREFILL and r.idle == [2, 4]
    assert r.c_prefill == 1.375 and r.c_decode == (0.125 + 0.5 + 0.0625) / 3


def test_extreme_scales_after_persisting():
    w = [1.0] + [0.0] * 7
    s = RefScheduler(params(w_prefill=w, scale_after=3), [PREFILL, DECODE])
    hot = [[5.0] + [0.0] * 11, [0.0] * 12]
    calm = [[0.0] * 12, [0.0] * 12]
    got = []
    for st in [hot, hot, hot, hot, calm, hot, hot, hot]:
        s.observe([st[0], st[1]])
        r = s.evaluate()
        got.append((r.scenario, r.scale_prefill, r.scale_decode))
    E, N = EXTREME, NORMAL
    assert got == [(E, 0, 0), (E, 0, 0), (E, 1, 0), (E, 0, 0), (N, 0, 0),
                   (E, 0, 0), (E, 0, 0), (E, 1, 0)]


@pytest.mark.parametrize("cp,cd,want", [
    (0.2499999, 0.2499999, LOW_LOAD),   # both under the lower thresholds
    (0.25, 0.0, NORMAL),                # strict: at the threshold is normal
    (0.0, -0.25, NORMAL),               # |C|
    (-0.1, 0.1, LOW_LOAD),
    (0.0, 1.5, IMBALANCED),             # one side low, the other busy: not low load
])
def test_low_load_boundaries(cp, cd, want):
    w = [1.0] + [0.0] * 7
    wd = [0.0, 0.0, 0.0, 0.0, 1.0, 0.0, 0.0, 0.0]   # C^d = T_b
    s = RefScheduler(params(w_prefill=w, w_decode=wd, eps_p_min=0.25, eps_d_min=0.25),
                     [PREFILL, DECODE])
    s.observe([[cp] + [0.0] * 11, [0.0] * 8 + [cd, 0.0, 0.0, 0.0]])
    assert s.evaluate().scenario == want


def test_low_load_is_off_at_zero_thresholds():
    s = RefScheduler(params(), [PREFILL, DECODE])
    s.observe([[0.0] * 12, [0.0] * 12])
    assert s.evaluate().scenario == NORMAL


def test_low_load_scales_down_after_persisting():
    """Two prefill nodes and one decode node, all quiet: on the third
    consecutive low-load evaluation the prefill side may give a node up; the
    decode side, with its only node, may not.  Normal load restarts the
    count; an overload run in between does not share it."""
    w = [1.0] + [0.0] * 7
    s = RefScheduler(params(w_prefill=w, scale_after=3, eps_p_min=0.5, eps_d_min=0.5),
                     [PREFILL, PREFILL, DECODE])
    quiet = [[0.0] * 12] * 3
    mid = [[0.75] + [0.0] * 11, [0.75] + [0.0] * 11, [0.0] * 12]    # C^p 0.75: normal
    hot = [[5.0] + [0.0] * 11, [5.0] + [0.0] * 11, [0.0] * 12]      # overload
    got = []
    for st in [quiet, quiet, quiet, quiet, mid, quiet, quiet, hot, quiet, quiet, quiet]:
        s.observe(st)
        r = s.evaluate()
        got.append((r.scenario, r.scale_prefill, r.scale_decode))
    L, N, E = LOW_LOAD, NORMAL, EXTREME
    assert got == [(L, 0, 0), (L, 0, 0), (L, -1, 0), (L, 0, 0), (N, 0, 0),
                   (L, 0, 0), (L, 0, 0), (E, 0, 0), (L, 0, 0), (L, 0, 0), (L, -1, 0)]


def test_offline_nodes_take_no_part():
    """An offline node's status counts in no average: with the busy node
    offline the averages are those of the others; it is never idle and never
    routed to."""
    w = [1.0] + [0.0] * 7
    wd = [0.0] * 4 + [1.0] + [0.0] * 3
    s = RefScheduler(params(w_prefill=w, w_decode=wd), [PREFILL, OFFLINE, DECODE])
    s.observe([[1.5] + [0.0] * 11, [9.0] * 12, [0.0] * 8 + [0.125, 0, 0, 0]])
    r = s.evaluate()
    assert (r.c_prefill, r.c_decode) == (1.5, 0.125)
    assert r.scenario == IMBALANCED and r.switch_to == PREFILL and r.idle == [2]
    roles = [PREFILL, OFFLINE, DECODE, OFFLINE]
    z = [[0.0] * 4] * 4
    assert route(roles, 100, [0] * 4, [0, 0, 0, 0], [1.0, 9.0, 1.0, 9.0], 1, z, z,
                 [9, 9, 9, 9]) == (0, 2)
    assert route([OFFLINE, DECODE], 100, [0, 0], [0, 0], [1.0, 1.0], 1, z, z, [9, 9]) == (-1, -1)


def brute_route(roles, prompt, hit, queued, rate, kv, spb, lat, free):
    """Every (P, D) pair, ordered by (TTFT of P, P) then (latency P->D, D)."""
    P = [i for i, r in enumerate(roles) if r == PREFILL and rate[i] > 0]
    D = [j for j, r in enumerate(roles) if r == DECODE and free[j] >= kv]
    if not P:
        return -1, -1
    pairs = []
    for i in P:
        ttft = (queued[i] + prompt - min(hit[i], prompt)) / rate[i]
        if not D:
            pairs.append(((ttft, i), (0.0, -1), i, -1))
        for j in D:
            pairs.append(((ttft, i), (lat[i][j] + kv * spb[i][j], j), i, j))
    best = min(pairs, key=lambda x: (x[0], x[1]))
    return best[2], best[3]


def test_route_matches_brute_force():
    rng = random.Random(7)
    for _ in range(400):
        n = rng.randint(1, 7)
        roles = [rng.choice([PREFILL, DECODE]) for _ in range(n)]
        prompt = rng.randint(1, 5000)
        hit = [rng.choice([0, rng.randint(0, 6000)]) for _ in range(n)]
        queued = [rng.randint(0, 20000) for _ in range(n)]
        rate = [rng.choice([0.0, 1000.0, 2000.0, 4000.0]) for _ in range(n)]
        kv = rng.randint(1, 1 << 30)
        spb = [[rng.choice([1e-9, 2e-9, 4e-11]) for _ in range(n)] for _ in range(n)]
        lat = [[rng.choice([1e-5, 1e-3]) for _ in range(n)] for _ in range(n)]
        free = [rng.choice([0, kv, 2 * kv]) for _ in range(n)]
        assert route(roles, prompt, hit, queued, rate, kv, spb, lat, free) == \
            brute_route(roles, prompt, hit, queued, rate, kv, spb, lat, free)


def test_route_closed_cases():
    roles = [PREFILL, PREFILL, DECODE, DECODE]
    spb = [[1e-9] * 4 for _ in range(4)]
    lat = [[0.0] * 4 for _ in range(4)]
    # node 1 holds the whole prompt in its prefix cache: only its queue counts
    p, d = route(roles, 1000, [0, 1000, 0, 0], [0, 500, 0, 0], [1000.0, 1000.0, 0, 0],
                 10, spb, lat, [0, 0, 100, 100])
    assert (p, d) == (1, 2)                       # 0.5 s against 1.0 s; tie on D -> lower
    # no decode node has room
    assert route(roles, 10, [0] * 4, [0] * 4, [1.0] * 4, 1000, spb, lat, [0, 0, 999, 0]) == (0, -1)
    # no prefill node
    assert route([DECODE, DECODE], 10, [0, 0], [0, 0], [1.0, 1.0], 1, spb, lat, [5, 5]) == (-1, -1)


def test_rejects_bad_parameters():
    with pytest.raises(ValueError):
        RefScheduler(params(window=0), [PREFILL])
    with pytest.raises(ValueError):
        RefScheduler(params(eps_p_high=0.5), [PREFILL])   # high below low
    with pytest.raises(ValueError):
        RefScheduler(params(scale=[1.0] * 11 + [0.0]), [PREFILL])
    with pytest.raises(ValueError):
        RefScheduler(params(), [3])                       # no such role (2 is offline)
    with pytest.raises(ValueError):
        RefScheduler(params(eps_p_min=1.5), [PREFILL])    # low-load threshold above low
    with pytest.raises(ValueError):
        RefScheduler(params(eps_d_min=-0.5), [PREFILL])
    s = RefScheduler(default_params(), [PREFILL, DECODE])
    with pytest.raises(ValueError):
        s.evaluate()                                      # nothing observed yet
    with pytest.raises(ValueError):
        s.observe([[0.0] * 12])                           # one vector per node


def test_scores_are_order_exact_sums():
    """Scores are plain float64 sums in the order of Algorithm 1's terms:
    adding the terms in that order with Python floats reproduces them bit
    for bit on random inputs (another implementation keeping the order, e.g.
    the native library, can therefore be compared exactly)."""
    rng = random.Random(3)
    p = default_params(window=3)
    for _ in range(50):
        s = RefScheduler(p, [PREFILL])
        hist = [[rng.uniform(0, 50) for _ in range(12)] for _ in range(rng.randint(1, 6))]
        for h in hist:
            s.observe([h])
        last = hist[-3:]
        norm = [sum(x[k] for x in last) / len(last) / p.scale[k] for k in range(12)]
        cp = 0.0
        for w, k in zip(p.w_prefill, [0, 1, 2, 3, 8, 9, 10, 11]):
            cp += w * norm[k]
        assert s.node_scores(0)[0] == cp
        assert all(itertools.starmap(lambda a, b: a == b, zip(s.smoothed(0), norm)))
