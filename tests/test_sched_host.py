"""The native load-aware scheduler (flowkv_sched_*) against the oracle, CPU.

Both sides evaluate Algorithm 1 in IEEE double in the same order, so the
scores must agree bit for bit and every decision (scenario, idle set, role
to take, scale requests, routing) exactly, on random parameters, status
streams and role changes.
"""

import random

import numpy as np
import pytest

from oracle.scheduler import (DECODE, LOW_LOAD, OFFLINE, PREFILL, Params, RefScheduler,
                              default_params, route)
from paper_2504_03775_amd import flowkv as fk


def to_native(p: Params):
    return fk.sched_params(p.window, p.scale, p.w_prefill, p.w_decode, p.eps_p_low, p.eps_d_low,
                           p.eps_p_high, p.eps_d_high, p.idle_threshold, p.scale_after,
                           p.eps_p_min, p.eps_d_min)


def random_params(rng: random.Random) -> Params:
    lo_p, lo_d = rng.uniform(0.05, 1.0), rng.uniform(0.05, 1.0)
    return Params(window=rng.randint(1, 9),
                  scale=[rng.choice([1.0, 3.0, 8.0, 64.0, 0.7]) for _ in range(12)],
                  w_prefill=[rng.uniform(0, 1) for _ in range(8)],
                  w_decode=[rng.uniform(0, 1) for _ in range(8)],
                  eps_p_low=lo_p, eps_d_low=lo_d,
                  eps_p_high=lo_p * rng.uniform(1, 3), eps_d_high=lo_d * rng.uniform(1, 3),
                  idle_threshold=rng.uniform(0, 0.5), scale_after=rng.randint(1, 4),
                  eps_p_min=rng.choice([0.0, lo_p * rng.uniform(0.1, 1.0)]),
                  eps_d_min=rng.choice([0.0, lo_d * rng.uniform(0.1, 1.0)]))


def drift(rng: random.Random, level: float) -> float:
    """A random walk of the status magnitude over four decades, so a run
    passes through low, normal, imbalanced and overloaded states."""
    return min(30.0, max(1e-4, level * rng.uniform(0.5, 1.8)))


@pytest.mark.parametrize("seed", range(40))
def test_evaluation_matches_oracle_exactly(seed):
    rng = random.Random(seed)
    p = random_params(rng)
    n = rng.randint(1, 12)
    roles = [rng.choice([PREFILL, DECODE, PREFILL, DECODE, OFFLINE]) for _ in range(n)]
    ref = RefScheduler(p, roles)
    nat = fk.Scheduler(to_native(p), roles)
    level = 10 ** rng.uniform(-3, 0.5)   # status magnitude: drifts through the scenarios
    seen = set()
    for step in range(60):
        level = drift(rng, level)
        status = [[rng.uniform(0, level) * (8.0 if k < 8 else 1.0) for k in range(12)]
                  for _ in range(n)]
        ref.observe(status)
        nat.observe(status)
        if rng.random() < 0.1:
            i, role = rng.randrange(n), rng.choice([PREFILL, DECODE, OFFLINE])
            ref.set_role(i, role)
            nat.set_role(i, role)
        want = ref.evaluate()
        got, idle, scores = nat.evaluate()
        seen.add(want.scenario)
        assert got.scenario == want.scenario, step
        assert got.c_prefill == want.c_prefill and got.c_decode == want.c_decode, step
        assert list(idle) == want.idle and got.switch_to == want.switch_to
        assert (got.scale_prefill, got.scale_decode) == (want.scale_prefill, want.scale_decode)
        for i in range(n):
            assert tuple(scores[i]) == ref.node_scores(i)
    assert seen  # every run covers at least one scenario; the set below covers all four


def test_all_scenarios_are_covered_by_the_random_runs():
    covered = set()
    for seed in range(40):
        rng = random.Random(seed)
        p = random_params(rng)
        n = rng.randint(1, 12)
        ref = RefScheduler(p, [rng.choice([PREFILL, DECODE, PREFILL, DECODE, OFFLINE])
                               for _ in range(n)])
        level = 10 ** rng.uniform(-3, 0.5)
        for _ in range(60):
            level = drift(rng, level)
            ref.observe([[rng.uniform(0, level) * (8.0 if k < 8 else 1.0) for k in range(12)]
                         for _ in range(n)])
            r = ref.evaluate()
            covered.add(r.scenario)
            if r.idle:
                covered.add("idle")
            if r.scale_prefill > 0 or r.scale_decode > 0:
                covered.add("scale up")
            if r.scale_prefill < 0 or r.scale_decode < 0:
                covered.add("scale down")
    assert covered >= {0, 1, 2, LOW_LOAD, "idle", "scale up", "scale down"}


@pytest.mark.parametrize("seed", range(10))
def test_routing_matches_oracle(seed):
    rng = random.Random(100 + seed)
    for _ in range(100):
        n = rng.randint(1, 9)
        roles = [rng.choice([PREFILL, DECODE, OFFLINE]) for _ in range(n)]
        nat = fk.Scheduler(to_native(default_params()), roles)
        prompt = rng.randint(0, 40000)
        hit = [rng.choice([0, rng.randint(-5, 50000)]) for _ in range(n)]
        queued = [rng.randint(0, 200000) for _ in range(n)]
        rate = [rng.choice([0.0, -1.0, 3000.0, 12000.0, 12000.5]) for _ in range(n)]
        kv = rng.randint(0, 1 << 34)
        spb = [[rng.choice([1e-9, 2.5e-10, 4.3e-11]) for _ in range(n)] for _ in range(n)]
        lat = [[rng.choice([0.0, 1e-5, 2e-3]) for _ in range(n)] for _ in range(n)]
        free = [rng.choice([0, kv, kv - 1, 1 << 40]) for _ in range(n)]
        assert nat.route(prompt, hit, queued, rate, kv, spb, lat, free) == \
            route(roles, prompt, hit, queued, rate, kv, spb, lat, free)


def test_errors():
    good = to_native(default_params())
    bad = [dict(window=0), dict(window=fk_max_window() + 1), dict(scale_after=0),
           dict(eps_p_low=0.0), dict(eps_d_high=0.1), dict(eps_p_high=float("inf")),
           dict(eps_p_min=-0.1), dict(eps_d_min=0.6), dict(eps_p_min=float("nan"))]
    for change in bad:
        p = to_native(default_params())
        for k, v in change.items():
            setattr(p, k, v)
        with pytest.raises(fk.FlowKVError) as e:
            fk.Scheduler(p, [PREFILL])
        assert e.value.code == fk.EINVAL, change
    p = to_native(default_params())
    p.scale[3] = 0.0
    with pytest.raises(fk.FlowKVError):
        fk.Scheduler(p, [PREFILL])
    with pytest.raises(fk.FlowKVError):
        fk.Scheduler(good, [PREFILL, 3])
    with pytest.raises(fk.FlowKVError):
        fk.Scheduler(good, [])
    s = fk.Scheduler(good, [PREFILL, DECODE])
    with pytest.raises(fk.FlowKVError) as e:
        s.evaluate()                                   # nothing observed yet
    assert e.value.code == fk.EINVAL
    with pytest.raises(fk.FlowKVError) as e:
        s.set_role(2, PREFILL)
    assert e.value.code == fk.ERANGE
    with pytest.raises(fk.FlowKVError):
        s.set_role(0, 5)
    s.set_role(0, OFFLINE)                             # a node can go offline and back
    s.set_role(0, PREFILL)
    with pytest.raises(ValueError):
        s.observe(np.zeros((3, 12)))
    z = [[0.0] * 2] * 2
    with pytest.raises(fk.FlowKVError):
        s.route(-1, [0, 0], [0, 0], [1.0, 1.0], 1, z, z, [1, 1])


def fk_max_window():
    import re
    import os
    text = open(os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                             "include", "flowkv.h")).read()
    return int(re.search(r"#define FLOWKV_SCHED_MAX_WINDOW (\d+)", text).group(1))
