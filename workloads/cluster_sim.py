"""A seeded discrete-event cluster of prefill (P) and decode (D) nodes that a
load-aware scheduler drives (the synthetic environment for section 3.4).

The paper evaluates its scheduler on a real cluster with unpublished weights;
this model stands in for that cluster.  It holds no part of the scheduler:
the caller passes a scheduler object (the native library's, or the oracle's
in the tests) with ``observe / evaluate / set_role / route``, and this module
only produces the status samples, applies the decisions and keeps time.

Model (all times in seconds):
* requests arrive as a Poisson stream; each has a prompt length and an
  output length drawn from the workload's mix;
* at arrival the scheduler routes the request to a prefill node and a decode
  node (Algorithm 1's routing); the decode node reserves the request's KV.
  A request no pair can take (no decode node with room) waits, in arrival
  order, and is routed again every scheduler period;
* a prefill node serves its queue first-in first-out at ``prefill_rate``
  tokens per second;
* the KV cache then moves to the decode node: latency + bytes / link rate,
  one transfer per request (the segment-coalesced transfer);
* a decode node runs continuous batching: each iteration costs
  ``iter_base + iter_per_req x batch + KV bytes read / kv_read_rate`` and
  gives every running request one token; requests join at iteration
  boundaries while the batch has room;
* every ``tick`` the scheduler observes each node's 12 status indicators
  (queue lengths, token budget, KV and GPU use over the last tick) and
  evaluates.  Under imbalanced load the idle nodes it names switch to the
  busier role once they hold no work of their old role (a role keeps at
  least one node).  Scale requests are counted; with ``scaling`` on, the
  model also applies them: a scale-up brings the lowest-indexed offline node
  online in the role asked for, and a scale-down takes the role's
  highest-indexed node offline once it has drained (a role keeps at least
  one node).  Offline nodes report zeros and take no requests; the model
  reports the node-seconds spent online (the cost that scaling down saves).
* arrivals may change rate over time (``phases``: consecutive (duration,
  rate) pieces), so one run can pass from busy to quiet and back.
"""

from __future__ import annotations

import heapq
import math
from collections import deque
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

PREFILL, DECODE, OFFLINE = 0, 1, 2
KV_BYTES_PER_TOKEN_8B = 32 * 2 * 8 * 128 * 2   # Llama-3-8B, bf16: 128 KiB per token


@dataclass
class ClusterConfig:
    roles: Sequence[int]
    prefill_rate: float = 40_000.0          # tokens/s per prefill node
    iter_base: float = 4e-3                 # decode iteration: fixed part
    iter_per_req: float = 5e-5              # per running request
    kv_read_rate: float = 5.4e12            # bytes/s of KV read per iteration
    max_batch: int = 128
    kv_capacity_tokens: int = 1_500_000     # per decode node
    link_rate: float = 50e9                 # bytes/s, one GPU-to-GPU link
    link_latency: float = 50e-6
    kv_bytes_per_token: int = KV_BYTES_PER_TOKEN_8B
    tick: float = 0.1                       # scheduler period
    switching: bool = True                  # apply idle-node role switches
    scaling: bool = False                   # apply scale-up / scale-down requests


@dataclass
class Workload:
    rate: float                             # arrivals per second
    n_requests: int
    prompts: Sequence[int]                  # prompt lengths, drawn uniformly
    outputs: Sequence[int]                  # output lengths, drawn uniformly
    seed: int = 0
    phases: Optional[Sequence[Tuple[float, float]]] = None  # (duration s, rate); then `rate`


# placeholder normalisation for the model's indicators (Algorithm 1 order)
STATUS_SCALE = [1, 8, 1, 8, 128, 32, 1, 8, 1, 1, 1, 1]


@dataclass
class _Req:
    rid: int
    arrival: float
    prompt: int
    output: int
    p: int = -1
    d: int = -1
    first_token: float = math.nan
    done: float = math.nan
    generated: int = 0


@dataclass
class _Node:
    role: int
    pending: Optional[int] = None           # role to take once drained
    queue: deque = field(default_factory=deque)
    busy: Optional[_Req] = None
    busy_until: float = 0.0
    sending: int = 0
    running: List[_Req] = field(default_factory=list)
    waiting: deque = field(default_factory=deque)
    iterating: bool = False
    reserved_tokens: int = 0
    busy_time: float = 0.0
    busy_since: Optional[float] = None


class Cluster:
    def __init__(self, cfg: ClusterConfig, sched):
        self.cfg = cfg
        self.sched = sched
        self.nodes = [_Node(role=r) for r in cfg.roles]
        self.n = len(self.nodes)
        self.now = 0.0
        self.events: list = []
        self.seq = 0
        self.log: List[tuple] = []          # (time, kind, ...) decisions, for comparisons
        self.done: List[_Req] = []
        self.switches = 0
        self.scale_requests = [0, 0]        # scale-ups asked: prefill, decode
        self.scale_downs = [0, 0]           # scale-downs asked: prefill, decode
        self.scenarios = [0, 0, 0, 0]       # normal, imbalanced, overload, low load
        self.node_seconds = 0.0             # time online, summed over nodes
        lat = [[cfg.link_latency] * self.n for _ in range(self.n)]
        spb = [[1.0 / cfg.link_rate] * self.n for _ in range(self.n)]
        self.lat, self.spb = lat, spb

    # ---- event plumbing ------------------------------------------------------
    def _at(self, t: float, kind: str, *payload) -> None:
        heapq.heappush(self.events, (t, self.seq, kind, payload))
        self.seq += 1

    def _set_busy(self, node: _Node, busy: bool) -> None:
        if busy and node.busy_since is None:
            node.busy_since = self.now
        elif not busy and node.busy_since is not None:
            node.busy_time += self.now - node.busy_since
            node.busy_since = None

    # ---- routing -------------------------------------------------------------
    def _route(self, req: _Req) -> None:
        cfg = self.cfg
        queued, rate, free = [], [], []
        for nd in self.nodes:
            q = sum(r.prompt for r in nd.queue)
            if nd.busy is not None:
                q += int(max(0.0, nd.busy_until - self.now) * cfg.prefill_rate)
            queued.append(q)
            active_p = nd.role == PREFILL and nd.pending is None
            rate.append(cfg.prefill_rate if active_p else 0.0)
            active_d = nd.role == DECODE and nd.pending is None
            room = cfg.kv_capacity_tokens - nd.reserved_tokens if active_d else 0
            free.append(room * cfg.kv_bytes_per_token)
        kv = (req.prompt + req.output) * cfg.kv_bytes_per_token
        p, d = self.sched.route(req.prompt, [0] * self.n, queued, rate, kv, self.spb, self.lat,
                                free)
        self.log.append((self.now, "route", req.rid, p, d))
        req.p, req.d = p, d
        if d >= 0:
            self.nodes[d].reserved_tokens += req.prompt + req.output

    # ---- prefill -------------------------------------------------------------
    def _start_prefill(self, i: int) -> None:
        nd = self.nodes[i]
        if nd.busy is not None or not nd.queue:
            return
        req = nd.queue.popleft()
        nd.busy = req
        nd.busy_until = self.now + req.prompt / self.cfg.prefill_rate
        self._set_busy(nd, True)
        self._at(nd.busy_until, "prefill_done", i)

    def _prefill_done(self, i: int) -> None:
        nd = self.nodes[i]
        req = nd.busy
        nd.busy = None
        self._set_busy(nd, False)
        req.first_token = self.now
        nd.sending += 1
        self._send(i, req)
        self._start_prefill(i)
        self._maybe_switch(i)

    def _send(self, i: int, req: _Req) -> None:
        cfg = self.cfg
        nbytes = req.prompt * cfg.kv_bytes_per_token
        t = cfg.link_latency + nbytes / cfg.link_rate
        self._at(self.now + t, "xfer_done", i, req)

    def _xfer_done(self, i: int, req: _Req) -> None:
        self.nodes[i].sending -= 1
        d = self.nodes[req.d]
        d.waiting.append(req)
        self._start_iter(req.d)

    # ---- decode --------------------------------------------------------------
    def _start_iter(self, j: int) -> None:
        nd, cfg = self.nodes[j], self.cfg
        if nd.iterating:
            return
        while nd.waiting and len(nd.running) < cfg.max_batch:
            nd.running.append(nd.waiting.popleft())
        if not nd.running:
            self._set_busy(nd, False)
            return
        kv_tokens = sum(r.prompt + r.generated for r in nd.running)
        t = (cfg.iter_base + cfg.iter_per_req * len(nd.running) +
             kv_tokens * cfg.kv_bytes_per_token / cfg.kv_read_rate)
        nd.iterating = True
        self._set_busy(nd, True)
        self._at(self.now + t, "iter_done", j)

    def _iter_done(self, j: int) -> None:
        nd = self.nodes[j]
        nd.iterating = False
        keep = []
        for r in nd.running:
            r.generated += 1
            if r.generated >= r.output:
                r.done = self.now
                nd.reserved_tokens -= r.prompt + r.output
                self.done.append(r)
            else:
                keep.append(r)
        nd.running = keep
        self._start_iter(j)
        self._maybe_switch(j)

    # ---- scheduler period ----------------------------------------------------
    def _status(self) -> List[List[float]]:
        cfg, out = self.cfg, []
        for nd in self.nodes:
            if nd.busy_since is not None:
                nd.busy_time += self.now - nd.busy_since
                nd.busy_since = self.now
            g = min(1.0, nd.busy_time / cfg.tick)
            nd.busy_time = 0.0
            s = [0.0] * 12
            if nd.role == OFFLINE:
                pass                            # an offline node reports zeros
            elif nd.role == PREFILL:
                s[0] = 1.0 if nd.busy is not None else 0.0
                s[1] = float(len(nd.queue))
                s[3] = float(nd.sending)
                s[8] = min(1.0, (sum(r.prompt for r in nd.queue) +
                                 (nd.busy.prompt if nd.busy else 0)) / (cfg.prefill_rate * cfg.tick))
                s[11] = 0.5 * g                 # prefill is compute-bound
            else:
                s[4] = float(len(nd.running))
                s[5] = float(len(nd.waiting))
                s[8] = len(nd.running) / cfg.max_batch
                s[9] = nd.reserved_tokens / cfg.kv_capacity_tokens
                s[11] = g                       # decode is bandwidth-bound
            s[10] = g
            out.append(s)
        return out

    def _tick(self) -> None:
        self.node_seconds += self.cfg.tick * sum(1 for nd in self.nodes if nd.role != OFFLINE)
        self.sched.observe(self._status())
        r = self.sched.evaluate()
        scen, idle, switch_to, sp, sd = r
        self.scenarios[scen] += 1
        for k, x in enumerate((sp, sd)):
            if x > 0:
                self.scale_requests[k] += x
            elif x < 0:
                self.scale_downs[k] -= x
        self.log.append((self.now, "eval", scen, tuple(idle), switch_to, sp, sd))
        if self.cfg.scaling:
            for role, x in ((PREFILL, sp), (DECODE, sd)):
                if x > 0:
                    self._scale_up(role)
                elif x < 0:
                    self._scale_down(role)
        if self.cfg.switching and idle:
            for i in idle:
                nd = self.nodes[i]
                # a role keeps at least one node: requests need both sides
                staying = sum(1 for x in self.nodes if x.role == nd.role and x.pending is None)
                if nd.role != switch_to and nd.pending is None and staying > 1:
                    nd.pending = switch_to
                    self._maybe_switch(i)
        # requests no node pair could take at arrival: route again, in order
        while self.backlog and self._admit(self.backlog[0]):
            self.backlog.popleft()
        if len(self.done) < self.total:
            self._at(self.now + self.cfg.tick, "tick")

    def _scale_up(self, role: int) -> None:
        for i, nd in enumerate(self.nodes):
            if nd.role == OFFLINE and nd.pending is None:
                nd.role = role
                self.sched.set_role(i, role)
                self.log.append((self.now, "online", i, role))
                return

    def _scale_down(self, role: int) -> None:
        active = [i for i, nd in enumerate(self.nodes) if nd.role == role and nd.pending is None]
        if len(active) > 1:
            i = active[-1]
            self.nodes[i].pending = OFFLINE
            self.log.append((self.now, "retire", i))
            self._maybe_switch(i)

    def _admit(self, req: _Req) -> bool:
        """Route a request; queue it at its prefill node if both sides exist."""
        self._route(req)
        if req.p < 0 or req.d < 0:
            if req.d >= 0:
                self.nodes[req.d].reserved_tokens -= req.prompt + req.output
            return False
        self.nodes[req.p].queue.append(req)
        self._start_prefill(req.p)
        return True

    def _maybe_switch(self, i: int) -> None:
        nd = self.nodes[i]
        if nd.pending is None:
            return
        drained = (nd.busy is None and not nd.queue) if nd.role == PREFILL else \
            (not nd.running and not nd.waiting and not nd.iterating and nd.reserved_tokens == 0)
        if drained:
            nd.role, nd.pending = nd.pending, None
            self.sched.set_role(i, nd.role)
            if nd.role == OFFLINE:
                self.log.append((self.now, "offline", i))
            else:
                self.switches += 1
                self.log.append((self.now, "switch", i, nd.role))

    # ---- driver --------------------------------------------------------------
    def run(self, wl: Workload, horizon: float = 3600.0) -> Dict[str, float]:
        rng = np.random.default_rng(wl.seed)
        gaps = rng.exponential(1.0, wl.n_requests)      # unit-rate gaps, scaled below
        prompts = rng.choice(np.asarray(wl.prompts), wl.n_requests)
        outputs = rng.choice(np.asarray(wl.outputs), wl.n_requests)
        # piecewise rates: phase j covers [ends[j-1], ends[j]); `rate` after
        ends, rates = [], []
        for dur, rate in (wl.phases or ()):
            ends.append((ends[-1] if ends else 0.0) + dur)
            rates.append(rate)
        t = 0.0
        for k in range(wl.n_requests):
            j = next((i for i, e in enumerate(ends) if t < e), None)
            t += float(gaps[k] * (1.0 / (rates[j] if j is not None else wl.rate)))
            self._at(t, "arrival", _Req(k, t, int(prompts[k]), int(outputs[k])))
        self.total = wl.n_requests
        self.backlog: deque = deque()
        self._at(0.0, "tick")
        while self.events:
            t, _, kind, payload = heapq.heappop(self.events)
            if t > horizon:
                break
            self.now = t
            if kind == "arrival":
                req = payload[0]
                if self.backlog or not self._admit(req):
                    self.backlog.append(req)
            elif kind == "prefill_done":
                self._prefill_done(*payload)
            elif kind == "xfer_done":
                self._xfer_done(*payload)
            elif kind == "iter_done":
                self._iter_done(*payload)
            elif kind == "tick":
                self._tick()
        return self.summary(wl)

    def summary(self, wl: Workload) -> Dict[str, float]:
        done = self.done
        if not done:
            return {"completed": 0}
        end = max(r.done for r in done)
        ttft = np.array([r.first_token - r.arrival for r in done])
        e2e = np.array([r.done - r.arrival for r in done])
        return {
            "completed": len(done),
            "makespan_s": end,
            "requests_per_s": len(done) / end,
            "output_tokens_per_s": sum(r.output for r in done) / end,
            "ttft_mean_s": float(ttft.mean()),
            "ttft_p99_s": float(np.percentile(ttft, 99)),
            "e2e_mean_s": float(e2e.mean()),
            "role_switches": self.switches,
            "scenario_ticks": list(self.scenarios),
            "scale_requests": list(self.scale_requests),
            "scale_downs": list(self.scale_downs),
            "node_seconds": round(self.node_seconds, 6),
        }


class NativeScheduler:
    """Adapter: the library's scheduler (paper_2504_03775_amd.flowkv.Scheduler)."""

    def __init__(self, fk, params, roles):
        self.s = fk.Scheduler(params, roles)

    def observe(self, status):
        self.s.observe(status)

    def evaluate(self):
        r, idle, _ = self.s.evaluate()
        return r.scenario, [int(x) for x in idle], r.switch_to, r.scale_prefill, r.scale_decode

    def set_role(self, i, role):
        self.s.set_role(i, role)

    def route(self, *args):
        return self.s.route(*args)
