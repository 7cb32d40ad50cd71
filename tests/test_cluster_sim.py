"""The load-aware scheduler inside the seeded cluster model (CPU).

* The whole simulation with the native scheduler equals, decision by decision,
  the same simulation with the oracle scheduler (every route, evaluation,
  idle set and role switch), on the three load mixes.
* Conservation: every request completes once, decode nodes end with no KV
  reserved, TTFT precedes completion.
* What Algorithm 1 is for: on a decode-heavy mix the idle prefill node takes
  the decode role and throughput rises over fixed roles; on a prefill-heavy
  mix the idle decode node takes the prefill role and TTFT falls; a balanced
  mix stays in normal load with no switch.
* The extreme scenarios' scaling, with the low-load reading on: a busy phase
  then a quiet one, on 2 prefill + 2 decode nodes and 2 offline spares.
  The cluster scales down when quiet and up when overloaded, native and
  oracle schedulers drive identical runs, every request completes, and the
  cluster spends fewer node-seconds than four fixed nodes.
"""

import pytest

from oracle.scheduler import Params, RefScheduler, route as ref_route
from paper_2504_03775_amd import flowkv as fk
from workloads.cluster_sim import (DECODE, OFFLINE, PREFILL, STATUS_SCALE, Cluster,
                                   ClusterConfig, NativeScheduler, Workload)

W = [0.25, 0.25, 0.125, 0.125, 0.0625, 0.0625, 0.0625, 0.0625]
PARAMS = dict(window=4, scale=STATUS_SCALE, w_prefill=W, w_decode=W, eps_p_low=0.5,
              eps_d_low=0.5, eps_p_high=1.0, eps_d_high=1.0, idle_threshold=0.1, scale_after=3)

MIXES = {
    "balanced": Workload(6.0, 160, [1000, 5000, 10000], [256], seed=1),
    "prefill-heavy": Workload(5.0, 150, [12000, 16000, 20000], [32], seed=2),
    "decode-heavy": Workload(30.0, 300, [500, 1000], [1024], seed=3),
}


# the same, with the low-load thresholds on
PARAMS_LOW = dict(PARAMS, eps_p_min=0.05, eps_d_min=0.05)
PHASED = Workload(0.5, 300, [1000, 4000, 8000], [128, 512], seed=4,
                  phases=((20.0, 12.0), (60.0, 0.5)))


class OracleScheduler:
    def __init__(self, roles, params=PARAMS):
        self.s = RefScheduler(Params(**params), roles)

    def observe(self, status):
        self.s.observe(status)

    def evaluate(self):
        r = self.s.evaluate()
        return r.scenario, r.idle, r.switch_to, r.scale_prefill, r.scale_decode

    def set_role(self, i, role):
        self.s.set_role(i, role)

    def route(self, prompt, hit, queued, rate, kv, spb, lat, free):
        return ref_route(self.s.roles, prompt, hit, queued, rate, kv, spb, lat, free)


def native(roles, p=PARAMS):
    return NativeScheduler(fk, fk.sched_params(p["window"], p["scale"], p["w_prefill"],
                                               p["w_decode"], p["eps_p_low"], p["eps_d_low"],
                                               p["eps_p_high"], p["eps_d_high"],
                                               p["idle_threshold"], p["scale_after"],
                                               p.get("eps_p_min", 0.0),
                                               p.get("eps_d_min", 0.0)), roles)


def simulate(mix, sched_factory, switching=True, roles=(PREFILL, PREFILL, DECODE, DECODE)):
    roles = list(roles)
    c = Cluster(ClusterConfig(roles=roles, switching=switching), sched_factory(roles))
    return c, c.run(MIXES[mix])


@pytest.mark.parametrize("mix", sorted(MIXES))
def test_native_and_oracle_schedulers_drive_identical_simulations(mix):
    cn, rn = simulate(mix, native)
    co, ro = simulate(mix, OracleScheduler)
    assert cn.log == co.log
    assert rn == ro


@pytest.mark.parametrize("mix", sorted(MIXES))
def test_conservation(mix):
    c, r = simulate(mix, native)
    wl = MIXES[mix]
    assert r["completed"] == wl.n_requests
    assert sorted(q.rid for q in c.done) == list(range(wl.n_requests))
    for q in c.done:
        assert q.arrival <= q.first_token <= q.done and q.generated == q.output
    for nd in c.nodes:
        assert nd.reserved_tokens == 0 and not nd.running and not nd.waiting and not nd.queue
    assert any(nd.role == PREFILL for nd in c.nodes) and any(nd.role == DECODE for nd in c.nodes)


def test_load_aware_switching_helps_imbalanced_mixes():
    _, fixed = simulate("decode-heavy", native, switching=False)
    cs, aware = simulate("decode-heavy", native, switching=True)
    assert aware["role_switches"] >= 1
    assert sum(nd.role == DECODE for nd in cs.nodes) == 3
    assert aware["requests_per_s"] > 1.1 * fixed["requests_per_s"]
    assert aware["e2e_mean_s"] < fixed["e2e_mean_s"]

    _, fixed = simulate("prefill-heavy", native, switching=False)
    cs, aware = simulate("prefill-heavy", native, switching=True)
    assert aware["role_switches"] >= 1
    assert sum(nd.role == PREFILL for nd in cs.nodes) == 3
    assert aware["ttft_mean_s"] < 0.9 * fixed["ttft_mean_s"]

    _, fixed = simulate("balanced", native, switching=False)
    _, aware = simulate("balanced", native, switching=True)
    assert aware == fixed and aware["role_switches"] == 0
    assert aware["scenario_ticks"][1] == aware["scenario_ticks"][2] == 0


def simulate_phased(sched_factory, roles, scaling):
    roles = list(roles)
    c = Cluster(ClusterConfig(roles=roles, switching=True, scaling=scaling), sched_factory(roles))
    return c, c.run(PHASED)


def test_scaling_with_low_load_native_equals_oracle():
    roles = (PREFILL, PREFILL, DECODE, DECODE, OFFLINE, OFFLINE)
    cn, rn = simulate_phased(lambda r: native(r, PARAMS_LOW), roles, True)
    co, ro = simulate_phased(lambda r: OracleScheduler(r, PARAMS_LOW), roles, True)
    assert cn.log == co.log
    assert rn == ro


def test_scaling_down_when_quiet_and_up_when_busy():
    roles = (PREFILL, PREFILL, DECODE, DECODE, OFFLINE, OFFLINE)
    c, r = simulate_phased(lambda x: native(x, PARAMS_LOW), roles, True)
    kinds = [e[1] for e in c.log]
    assert "offline" in kinds and "online" in kinds
    assert r["scenario_ticks"][3] > 0 and r["scale_downs"][0] >= 1 and r["scale_requests"][0] >= 1
    # every scale-down took a node offline only after it drained, and a role
    # always kept a node: replay the role changes
    now = list(roles)
    for e in c.log:
        if e[1] == "offline":
            now[e[2]] = OFFLINE
        elif e[1] in ("online", "switch"):
            now[e[2]] = e[3]
        assert PREFILL in now and DECODE in now
    assert r["completed"] == PHASED.n_requests
    for nd in c.nodes:
        assert nd.reserved_tokens == 0 and not nd.running and not nd.queue
    # four fixed nodes (no scaling, no spares) serve the same stream
    _, fixed = simulate_phased(native, (PREFILL, PREFILL, DECODE, DECODE), False)
    assert fixed["completed"] == PHASED.n_requests
    assert r["node_seconds"] < 0.7 * fixed["node_seconds"]


def test_low_load_off_leaves_the_fixed_runs_unchanged():
    """With the lower thresholds at 0 the scheduler never reports low load,
    and a run with scaling on but no overload equals the run with it off."""
    c1, r1 = simulate("balanced", native)
    assert r1["scenario_ticks"][3] == 0 and r1["scale_downs"] == [0, 0]
    roles = [PREFILL, PREFILL, DECODE, DECODE]
    c2 = Cluster(ClusterConfig(roles=roles, scaling=True), native(roles))
    assert c2.run(MIXES["balanced"]) == r1 and c2.log == c1.log
