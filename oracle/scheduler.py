"""Oracle for the Load-Aware Scheduler (test infrastructure only).

FlowKV (arXiv 2504.03775), section 3.4 and Appendix A (Algorithm 1, the node
status indicators): every node reports a status vector S_i; the controller
smooths it over a sliding window, normalises it, forms a prefill score C_i^p
and a decode score C_i^d as weighted sums, averages them over the prefill and
the decode nodes (C^p, C^d) and compares the averages with thresholds to
pick the scenario:

    low load    |C^p| <  eps_p_min  and |C^d| <  eps_d_min    (an extreme case)
    normal      |C^p| <= eps_p_low  and |C^d| <= eps_d_low    (otherwise)
    imbalanced  |C^p| <= eps_p_high and |C^d| <= eps_d_high   (otherwise)
    extreme     anything else (overload)

Normal load routes a request to the prefill node with the smallest
time-to-first-token given its prefix-cache hit, then to the decode node with
the smallest transfer latency from that prefill node.  Imbalanced load names
the idle nodes (score below a threshold) so their hybrid schedulers take the
busier role.  Extreme load that lasts asks for more nodes (overload) or for
fewer (low load).  Section 3.4 counts both system overload and low load as
extreme scenarios, and Appendix A's extreme-load paragraph scales up or,
conversely, down once the scores have lasted; Algorithm 1's own branches
test only the upper thresholds, under which low load would read as normal.
The reading here adds the lower pair (eps_p_min, eps_d_min), tested first;
0 turns it off.  Nodes may also be offline (a third role): they report
status but take part in no average, no idle set and no route.

The paper leaves the window, the normalisation, the weights, the thresholds,
the TTFT and latency models and the role an idle node takes unstated; this
module takes the readings written beside each step (they are also listed
with the other readings of the paper in the design notes).  Everything is
float64, evaluated term by term in the order written, so another
implementation that keeps that order agrees bit for bit.

Status vector order (Algorithm 1):
    0 L_r^p   1 L_w^p   2 L_sw^p   3 L_se^p      prefill queues
    4 L_r^d   5 L_w^d   6 L_sw^d   7 L_se^d      decode queues
    8 T_b     9 KV_u   10 G_u     11 MB_u        shared
Weights per role, in the order of the score's terms:
    w_r, w_w, w_sw, w_se, w_t, w_kv, w_g, w_mb

Parity: the steps Algorithm 1 states are pinned in
``tests/test_oracle_scheduler.py``:
- one-hot weights read the indicator each term names;
- window closed forms (a constant passes through; a spike leaves after
  exactly ``window`` samples; a ramp's mean);
- averages over own-role nodes only;
- hand-worked scenario boundaries, idle sets and the persistence of
  extreme load;
- routing against brute force over every (prefill, decode) pair;
- low load: strict lower thresholds tested first, its own persistence count,
  scale-down only for roles with more than one node, offline nodes in no
  average, idle set or route, all worked by hand.

The readings themselves (window, normalisation, weights, thresholds, the
TTFT and latency models, the idle node's new role, the low-load thresholds
and the scale-down rule) are **parity unpinned**: the paper prints no example
or number to check them against.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Sequence, Tuple

N_IND = 12
PREFILL, DECODE, OFFLINE = 0, 1, 2
NORMAL, IMBALANCED, EXTREME, LOW_LOAD = 0, 1, 2, 3

# the indicators each role's score reads, in the order of its weights
TERMS = {PREFILL: (0, 1, 2, 3, 8, 9, 10, 11), DECODE: (4, 5, 6, 7, 8, 9, 10, 11)}


@dataclass
class Params:
    window: int                     # samples in the sliding window
    scale: Sequence[float]          # 12 normalisation divisors
    w_prefill: Sequence[float]      # 8 weights of C^p
    w_decode: Sequence[float]       # 8 weights of C^d
    eps_p_low: float
    eps_d_low: float
    eps_p_high: float
    eps_d_high: float
    idle_threshold: float
    scale_after: int                # consecutive extreme evaluations before scaling
    eps_p_min: float = 0.0          # low load: both averages below these (0: never)
    eps_d_min: float = 0.0


@dataclass
class Result:
    scenario: int
    c_prefill: float
    c_decode: float
    idle: List[int] = field(default_factory=list)
    switch_to: int = -1             # role the idle nodes take (imbalanced), else -1
    scale_prefill: int = 0          # +1: the prefill side asks for another node,
    scale_decode: int = 0           # -1: it can give one up (low load)


class RefScheduler:
    """Algorithm 1, one evaluation per call, in plain Python."""

    def __init__(self, p: Params, roles: Sequence[int]):
        if p.window < 1 or len(p.scale) != N_IND or any(s <= 0 for s in p.scale):
            raise ValueError("bad window or normalisation")
        if len(p.w_prefill) != 8 or len(p.w_decode) != 8 or p.scale_after < 1:
            raise ValueError("bad weights or scale_after")
        if not (0 < p.eps_p_low <= p.eps_p_high and 0 < p.eps_d_low <= p.eps_d_high):
            raise ValueError("thresholds need 0 < low <= high")
        if not (0 <= p.eps_p_min <= p.eps_p_low and 0 <= p.eps_d_min <= p.eps_d_low):
            raise ValueError("low-load thresholds need 0 <= min <= low")
        if any(r not in (PREFILL, DECODE, OFFLINE) for r in roles) or not roles:
            raise ValueError("roles must be PREFILL, DECODE or OFFLINE")
        self.p = p
        self.roles = list(roles)
        self.history: List[List[List[float]]] = [[] for _ in roles]  # per node: samples
        self.extreme_run = 0        # consecutive overload evaluations
        self.low_run = 0            # consecutive low-load evaluations

    def set_role(self, node: int, role: int) -> None:
        if role not in (PREFILL, DECODE, OFFLINE):
            raise ValueError("bad role")
        self.roles[node] = role

    def observe(self, status: Sequence[Sequence[float]]) -> None:
        """One sample of S_i for every node (Algorithm 1: update the status)."""
        if len(status) != len(self.roles):
            raise ValueError("one status vector per node")
        for i, s in enumerate(status):
            if len(s) != N_IND:
                raise ValueError("12 indicators per node")
            self.history[i].append([float(x) for x in s])
            if len(self.history[i]) > self.p.window:
                self.history[i].pop(0)

    # Reading: the sliding window is the mean of the last `window` samples
    # (fewer before the window has filled); normalisation divides each
    # indicator by its configured scale.
    def smoothed(self, i: int) -> List[float]:
        h = self.history[i]
        if not h:
            raise ValueError("no sample observed yet")
        out = []
        for k in range(N_IND):
            acc = 0.0
            for sample in h:
                acc += sample[k]
            out.append(acc / len(h) / self.p.scale[k])
        return out

    def node_scores(self, i: int) -> Tuple[float, float]:
        """C_i^p and C_i^d of Algorithm 1: weighted sums, term by term."""
        s = self.smoothed(i)
        cp = 0.0
        for w, k in zip(self.p.w_prefill, TERMS[PREFILL]):
            cp += w * s[k]
        cd = 0.0
        for w, k in zip(self.p.w_decode, TERMS[DECODE]):
            cd += w * s[k]
        return cp, cd

    def evaluate(self) -> Result:
        p = self.p
        scores = [self.node_scores(i) for i in range(len(self.roles))]
        # C^p over the N prefill nodes, C^d over the M decode nodes (a role
        # with no node averages to 0)
        sp, n = 0.0, 0
        sd, m = 0.0, 0
        for i, role in enumerate(self.roles):
            if role == PREFILL:
                sp += scores[i][0]
                n += 1
            elif role == DECODE:
                sd += scores[i][1]
                m += 1
        cp = sp / n if n else 0.0
        cd = sd / m if m else 0.0
        # Reading: low load -- both averages under their lower thresholds --
        # is the extreme scenario's other side; once it has lasted
        # scale_after evaluations each role with more than one node may give
        # one up
        if abs(cp) < p.eps_p_min and abs(cd) < p.eps_d_min:
            self.extreme_run = 0
            self.low_run += 1
            r = Result(LOW_LOAD, cp, cd)
            if self.low_run >= p.scale_after:
                r.scale_prefill = -int(n > 1)
                r.scale_decode = -int(m > 1)
                self.low_run = 0
            return r
        self.low_run = 0
        if abs(cp) <= p.eps_p_low and abs(cd) <= p.eps_d_low:
            self.extreme_run = 0
            return Result(NORMAL, cp, cd)
        if abs(cp) <= p.eps_p_high and abs(cd) <= p.eps_d_high:
            self.extreme_run = 0
            # Reading: a node is idle when the score of its own role is below
            # the threshold; idle nodes of the less loaded side take the role
            # of the busier side (the side with the larger average score
            # relative to its low threshold)
            busier = PREFILL if cp / p.eps_p_low >= cd / p.eps_d_low else DECODE
            idle = [i for i, role in enumerate(self.roles)
                    if role not in (busier, OFFLINE) and scores[i][role] < p.idle_threshold]
            return Result(IMBALANCED, cp, cd, idle, busier)
        # Reading: extreme load asks for another node of each side beyond its
        # high threshold once the scenario has lasted scale_after evaluations
        self.extreme_run += 1
        r = Result(EXTREME, cp, cd)
        if self.extreme_run >= p.scale_after:
            r.scale_prefill = int(abs(cp) > p.eps_p_high)
            r.scale_decode = int(abs(cd) > p.eps_d_high)
            self.extreme_run = 0
        return r


def route(roles: Sequence[int], prompt_tokens: int, prefix_hit: Sequence[int],
          queued_tokens: Sequence[int], prefill_rate: Sequence[float], kv_bytes: int,
          xfer_sec_per_byte: Sequence[Sequence[float]], xfer_latency: Sequence[Sequence[float]],
          free_bytes: Sequence[int]) -> Tuple[int, int]:
    """Normal-load routing (Algorithm 1).

    Reading: TTFT on prefill node i is (queued prefill tokens + the prompt's
    tokens not covered by i's prefix cache) / i's prefill rate; the prefill
    node is the one with the smallest TTFT.  The transfer latency to decode
    node j is latency[P][j] + kv_bytes * sec_per_byte[P][j]; the decode node
    is the one with the smallest latency among those with kv_bytes free.
    Ties go to the lower node index.  Returns (P_t, D_t), -1 where no node
    qualifies."""
    best_p, best_t = -1, 0.0
    for i, role in enumerate(roles):
        if role != PREFILL or prefill_rate[i] <= 0:
            continue
        uncached = prompt_tokens - min(prefix_hit[i], prompt_tokens)
        t = (queued_tokens[i] + uncached) / prefill_rate[i]
        if best_p < 0 or t < best_t:
            best_p, best_t = i, t
    if best_p < 0:
        return -1, -1
    best_d, best_l = -1, 0.0
    for j, role in enumerate(roles):
        if role != DECODE or free_bytes[j] < kv_bytes:
            continue
        lat = xfer_latency[best_p][j] + kv_bytes * xfer_sec_per_byte[best_p][j]
        if best_d < 0 or lat < best_l:
            best_d, best_l = j, lat
    return best_p, best_d


def default_params(window: int = 4) -> Params:
    """Placeholder weights and thresholds (the paper's are unpublished):
    queue lengths and utilisations weigh equally, the token budget counts
    half; thresholds on the normalised scale."""
    return Params(window=window,
                  scale=[8, 32, 8, 8, 64, 64, 8, 8, 1, 1, 1, 1],
                  w_prefill=[0.25, 0.25, 0.125, 0.125, 0.0625, 0.0625, 0.0625, 0.0625],
                  w_decode=[0.25, 0.25, 0.125, 0.125, 0.0625, 0.0625, 0.0625, 0.0625],
                  eps_p_low=0.5, eps_d_low=0.5, eps_p_high=1.0, eps_d_high=1.0,
                  idle_threshold=0.1, scale_after=3)
