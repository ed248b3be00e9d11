"""TOPAS prefix-state scheduling (Sec. 4): the host-side decision that picks
which agent prefixes stay resident and which requests run under them.

At a scheduling event the GPU state is S_t = (R_t, Q_t): resident agent
prefixes and running requests (Sec. 3).  A decision picks a post-decision
state S' = (R', Q') with R' the agents of Q' (no idle prefixes) inside the
KV budget of Eq. (2):

    sum_{a in R'} l_a + sum_{r in Q'} d_r <= B_t.

Candidates are scored by Eq. (13),

    Score = J_admit^age - J_move - J_redo - J_revoke + V_reuse,

where J_admit^age sums, over the admitted requests A in their greedy order,
the task's age weight g_i(t) (Eq. (12)) times the request's conditional
progress Delta_task (Eq. (6)): the drop in the task's expected longest
remaining LLM-service path (Eq. (5)) over the workflow DAG, with every
unfinished stage's residual drawn from its empirical profile conditioned on
the service already recorded (Eq. (4)) and the hypothetical completion of a
request cutting its stage's residual by the request's expected service.
J_move charges the serialized prefix transfers (Eq. (8)) once per admitted
task waiting for an incoming prefix, J_redo the decode work a preemption
discards (Eq. (9)), J_revoke the credit granted to preempted requests at
their admission (Eq. (10)), and V_reuse values keeping prefixes that
downstream stages about to become ready will use (Eq. (11)).

Candidates come from GreedyPack over prefix sets (Sec. 4.5): every subset of
the active agents when there are at most M of them, else a greedy search
from R_t with single additions, one round of pair additions and drop/swap
repairs (Alg. 1).  The highest-scoring candidate wins (Eq. (14)), with
deterministic ties.

Readings where the paper is silent (the supplementary material that fixes
them is not available): see ``Params`` for beta, rho, H_age, M and K, and
the tie rules at ``_state_key``.  A started stage whose recorded service
already reaches every profile sample has residual 0.  A request's expected
service D-hat is an input (measured tables or history supply it).

The scenario a decision reads is a plain dict (see ``workflows.py`` for the
generator and the format); the decision is a ``Decision``.

Product side: numpy only; no device work.
"""

from __future__ import annotations

import itertools
import math
from dataclasses import dataclass, field

import numpy as np

# Two scores closer than this (relative to max(1, |score|)) are a tie.
TIE_RTOL = 1e-9
# Largest joint residual support enumerated for one task's expectation.
MAX_JOINT_SUPPORT = 1 << 22


@dataclass(frozen=True)
class Params:
    """Scheduler constants.  budget (B_t) is in tokens; mu in bytes per
    prefix token; b_swap in bytes per second; t_decode in seconds per decode
    token.  beta (Eq. (11)), rho and h_age (Eq. (12)), M and K (Alg. 1) are
    not given in the paper; the defaults are this build's readings."""
    budget: float
    mu: float
    b_swap: float
    t_decode: float
    beta: float = 0.5
    rho: float = 0.5
    h_age: float = 1.0
    M: int = 6
    K: int = 0


@dataclass
class Decision:
    resident: tuple            # R', sorted agent ids
    running: tuple             # Q', sorted request ids
    admitted: list             # A, request ids in greedy order
    preempted: tuple           # P, sorted request ids
    score: float
    credits: dict = field(default_factory=dict)   # lambda_r of each admitted request (Eq. (10))
    candidates: int = 0        # candidate states scored


# --------------------------------------------------------------------------- expected remaining path

class _TaskPaths:
    """One task's unfinished stages as arrays: each stage's residual support
    and probabilities (Eq. (4)), and the expected longest remaining path
    under any per-stage reductions (Eq. (5)), memoised."""

    def __init__(self, dag, task, profiles):
        self.order = dag["topo"]            # stages, predecessors first
        self.succ = dag["succ"]
        self.supports = {}                  # stage -> (values, probs)
        for v, st in enumerate(task["stages"]):
            status = st["status"]
            if status == "done":
                continue
            x = np.asarray(profiles[v], dtype=np.float64)
            e = float(st.get("served", 0.0))
            if e > 0.0:
                x = x[x > e] - e            # X - e given X > e
                if x.size == 0:
                    continue                # profile exhausted: nothing left
            vals, counts = np.unique(x, return_counts=True)
            self.supports[v] = (vals, counts / counts.sum())
        size = 1
        for vals, _ in self.supports.values():
            size *= vals.size
        if size > MAX_JOINT_SUPPORT:
            raise ValueError(f"joint residual support of {size} points is too large to enumerate")
        self.stages = sorted(self.supports)
        self.axis = {v: i for i, v in enumerate(self.stages)}
        probs = np.ones(())
        for v in self.stages:
            p = self.supports[v][1]
            probs = np.multiply.outer(probs, p)
        self.probs = probs
        self.memo = {}

    def expected_lp(self, cut):
        """E[LP] with stage v's residual replaced by [Z_v - cut[v]]_+."""
        key = tuple(sorted((v, c) for v, c in cut.items() if c > 0.0 and v in self.supports))
        hit = self.memo.get(key)
        if hit is not None:
            return hit
        nd = len(self.stages)
        cut = dict(key)
        z = {}
        for v in self.stages:
            vals = np.maximum(self.supports[v][0] - cut.get(v, 0.0), 0.0)
            shape = [1] * nd
            shape[self.axis[v]] = vals.size
            z[v] = vals.reshape(shape)
        # Longest path from each stage to a sink, in reverse topological order.
        lp = {}
        best = np.zeros([1] * nd) if nd else np.zeros(())
        for v in reversed(self.order):
            tail = None
            for w in self.succ[v]:
                tail = lp[w] if tail is None else np.maximum(tail, lp[w])
            own = z.get(v, 0.0)
            lp[v] = own if tail is None else own + tail
            best = np.maximum(best, lp[v])
        val = float(np.sum(np.broadcast_to(best, self.probs.shape) * self.probs)) if nd else 0.0
        self.memo[key] = val
        return val


# --------------------------------------------------------------------------- the scheduler

class TopasScheduler:
    """Decides one scheduling event from a scenario dict (see workflows.py)."""

    def __init__(self, scenario, params: Params):
        self.sc = scenario
        self.p = params
        dag = scenario["dag"]
        n = len(dag["agent"])
        succ = [[] for _ in range(n)]
        pred = [[] for _ in range(n)]
        for u, v in dag["edges"]:
            succ[u].append(v)
            pred[v].append(u)
        topo, seen = [], [False] * n

        def visit(v):
            if seen[v]:
                return
            seen[v] = True
            for u in pred[v]:
                visit(u)
            topo.append(v)

        for v in range(n):
            visit(v)
        self.dag = {"topo": topo, "succ": succ, "pred": pred, "agent": list(dag["agent"])}
        self.plen = {int(a): int(l) for a, l in enumerate(scenario["prefix_len"])}
        self.now = float(scenario["now"])
        self.tasks = {int(t["id"]): t for t in scenario["tasks"]}
        self.paths = {tid: _TaskPaths(self.dag, t, scenario["profiles"]) for tid, t in self.tasks.items()}
        self.req = {int(r["id"]): r for r in scenario["requests"]}
        self.running = sorted(r for r, q in self.req.items() if q["running"])
        self.waiting = sorted(r for r, q in self.req.items() if not q["running"])
        self.r_t = frozenset(int(a) for a in scenario["resident"])
        self.age = {tid: 1.0 + params.rho * math.log1p((self.now - float(t["arrival"])) / params.h_age)
                    for tid, t in self.tasks.items()}
        self.n_next = self._downstream_counts()
        self.evaluated = 0

    # ---- terms ----
    def agent_of(self, r):
        return self.dag["agent"][self.req[r]["stage"]]

    def _downstream_counts(self):
        """n_a(t) of Eq. (11): stages of agent a not yet started whose only
        unfinished predecessor is running."""
        n = {}
        for t in self.tasks.values():
            st = t["stages"]
            for w, s in enumerate(st):
                if s["status"] != "pending":
                    continue
                open_pred = [u for u in self.dag["pred"][w] if st[u]["status"] != "done"]
                if len(open_pred) == 1 and st[open_pred[0]]["status"] == "running":
                    a = self.dag["agent"][w]
                    n[a] = n.get(a, 0) + 1
        return n

    def progress(self, r, cut):
        """Delta_task (Eq. (6)) of request r after the reductions ``cut``
        already granted to its task's stages; returns (delta, new cut)."""
        q = self.req[r]
        paths = self.paths[int(q["task"])]
        v = int(q["stage"])
        after = dict(cut)
        after[v] = after.get(v, 0.0) + float(q["d_hat"])
        return paths.expected_lp(cut) - paths.expected_lp(after), after

    def move_time(self, r_new):
        r_in, r_out = r_new - self.r_t, self.r_t - r_new
        tokens = sum(self.plen[a] for a in r_out) + sum(self.plen[a] for a in r_in)
        return self.p.mu / self.p.b_swap * tokens

    def reuse_value(self, r_new):
        return self.p.beta * sum(self.n_next.get(a, 0) * self.p.mu * self.plen[a] / self.p.b_swap for a in r_new)

    def score(self, r_new, admitted, gains, preempted):
        """Eq. (13) of the state (r_new, running after the decision);
        ``gains`` are the admitted requests' g * Delta in greedy order."""
        r_in = r_new - self.r_t
        waiting_tasks = {int(self.req[r]["task"]) for r in admitted if self.agent_of(r) in r_in}
        j_move = self.move_time(r_new) * len(waiting_tasks)
        j_redo = sum(self.p.t_decode * float(self.req[r].get("generated", 0)) for r in preempted)
        j_revoke = sum(float(self.req[r].get("credit", 0.0)) for r in preempted)
        return sum(gains) - j_move - j_redo - j_revoke + self.reuse_value(r_new)

    # ---- GreedyPack ----
    def greedy_pack(self, r_set):
        """States for prefix set r_set (Sec. 4.5): running requests it covers
        stay, the others are preempted; then the fitting request with the
        largest g * Delta per KV token is admitted, one at a time, keeping
        room (capacity and an admission slot) for one request of every agent
        of r_set not yet covered.  Every intermediate allocation covering
        r_set is emitted.  Returns a list of (score, key, state) tuples."""
        p = self.p
        r_set = frozenset(r_set)
        keep = [r for r in self.running if self.agent_of(r) in r_set]
        preempted = tuple(r for r in self.running if self.agent_of(r) not in r_set)
        if p.K and len(preempted) > p.K:
            return []
        covered = {self.agent_of(r) for r in keep}
        pool = {a: [] for a in r_set}
        for r in self.waiting:
            a = self.agent_of(r)
            if a in pool:
                pool[a].append(r)
        reserve = {}
        for a in r_set - covered:
            if not pool[a]:
                return []                       # r_set cannot be covered
            reserve[a] = min(float(self.req[r]["d"]) for r in pool[a])
        used = sum(self.plen[a] for a in r_set) + sum(float(self.req[r]["d"]) for r in keep)
        if used + sum(reserve.values()) > p.budget:
            return []
        if p.K and len(reserve) > p.K:
            return []
        admitted, gains, credits = [], [], {}
        cuts = {}                                 # task -> stage reductions granted so far
        represented = {int(self.req[r]["task"]) for r in keep}
        out = []

        def emit():
            if reserve:
                return
            running = tuple(sorted(keep + admitted))
            s = self.score(r_set, admitted, gains, preempted)
            state = Decision(tuple(sorted(r_set)), running, list(admitted), preempted, s, dict(credits))
            out.append((s, _state_key(state, self.r_t), state))

        emit()
        left = [r for a in sorted(r_set) for r in pool[a]]
        while left and not (p.K and len(admitted) >= p.K):
            best = None
            for r in left:
                a = self.agent_of(r)
                d = float(self.req[r]["d"])
                need = sum(v for b, v in reserve.items() if b != a)
                if used + d + need > p.budget:
                    continue
                if p.K and len(admitted) + 1 + sum(1 for b in reserve if b != a) > p.K:
                    continue
                task = int(self.req[r]["task"])
                delta, _ = self.progress(r, cuts.get(task, {}))
                rate = self.age[task] * delta / max(d, 1.0)
                cand = (rate, task in represented, -r)
                if best is None or _better_rate(cand, best[0]):
                    best = (cand, r, delta)
            if best is None:
                break
            _, r, delta = best
            task = int(self.req[r]["task"])
            _, cuts[task] = self.progress(r, cuts.get(task, {}))
            left.remove(r)
            admitted.append(r)
            g = self.age[task] * delta
            gains.append(g)
            credits[r] = g
            represented.add(task)
            used += float(self.req[r]["d"])
            reserve.pop(self.agent_of(r), None)
            emit()
        self.evaluated += len(out)
        return out

    def phi(self, states):
        return max((s for s, _, _ in states), default=-math.inf)

    # ---- Alg. 1 ----
    def decide(self) -> Decision:
        p = self.p
        active = sorted({self.agent_of(r) for r in self.waiting + self.running})
        cand = []
        if len(active) <= p.M:
            for k in range(len(active) + 1):
                for sub in itertools.combinations(active, k):
                    cand += self.greedy_pack(sub)
        else:
            r_g = self.r_t
            cand += self.greedy_pack(r_g)
            for rs in self._repairs(r_g, active):
                cand += self.greedy_pack(rs)
            phi_g = self.phi(self.greedy_pack(r_g))
            tried_pairs = False
            while True:
                best = None
                for a in active:
                    if a in r_g:
                        continue
                    st = self.greedy_pack(r_g | {a})
                    cand += st
                    f = self.phi(st)
                    if best is None or _improves(f, best[0]):
                        best = (f, r_g | {a})
                if best is not None and _improves(best[0], phi_g):
                    r_g, phi_g = best[1], best[0]
                    continue
                if tried_pairs:
                    break
                tried_pairs = True
                best = None
                rest = [a for a in active if a not in r_g]
                for a, b in itertools.combinations(rest, 2):
                    st = self.greedy_pack(r_g | {a, b})
                    cand += st
                    f = self.phi(st)
                    if best is None or _improves(f, best[0]):
                        best = (f, r_g | {a, b})
                if best is not None and _improves(best[0], phi_g):
                    r_g, phi_g = best[1], best[0]
                    continue
                break
            for rs in self._repairs(r_g, active):
                cand += self.greedy_pack(rs)
            inc = Decision(tuple(sorted(self.r_t)), tuple(self.running), [], (),
                           self.score(self.r_t, [], [], ()), {})
            cand.append((inc.score, _state_key(inc, self.r_t), inc))
        if not self.running and any(st.running for _, _, st in cand):
            cand = [c for c in cand if c[2].running]
        if not cand:
            raise RuntimeError("no feasible state")
        best = cand[0]
        for c in cand[1:]:
            if _better_state(c, best):
                best = c
        out = best[2]
        out.candidates = len(cand)
        return out

    def _repairs(self, r_set, active):
        """Single-agent drops and swaps of r_set."""
        r_set = frozenset(r_set)
        out = []
        for a in sorted(r_set):
            out.append(r_set - {a})
            for b in active:
                if b not in r_set:
                    out.append((r_set - {a}) | {b})
        return out


def _tol(x):
    return TIE_RTOL * max(1.0, abs(x))


def _improves(new, old):
    if old == -math.inf:
        return new > -math.inf
    return new > old + _tol(old)


def _better_rate(a, b):
    """Greedy order: larger rate; within a tie, a request of a task already
    represented; then the lower request id."""
    if abs(a[0] - b[0]) > _tol(b[0]):
        return a[0] > b[0]
    return (a[1], a[2]) > (b[1], b[2])


def _state_key(st: Decision, r_t):
    """Tie order between equal scores (Eq. (14)'s deterministic ties): fewer
    preemptions, then fewer prefixes moved, then the lexicographically
    smaller resident set, then the smaller running set."""
    moved = len(set(st.resident) ^ set(r_t))
    return (len(st.preempted), moved, st.resident, st.running)


def _better_state(a, b):
    if abs(a[0] - b[0]) > _tol(b[0]):
        return a[0] > b[0]
    return a[1] < b[1]


def decide(scenario, params: Params) -> Decision:
    return TopasScheduler(scenario, params).decide()
