"""Plain reference of the TOPAS scheduling decision (Sec. 4, Eq. (3)-(14),
GreedyPack and Alg. 1).

TEST INFRASTRUCTURE ONLY: imported by tests, never by the product path.

The steps follow the paper's order and notation, in slow and direct code:

  * Eq. (4): a started stage's residual is its empirical profile X
    conditioned on X > e (the service recorded so far), shifted by -e; an
    unstarted stage's residual is X; a finished stage's is 0.
  * Eq. (5): L_i(H) = E[LP(G, Z_i(H))], the expectation over every joint
    realization of the unfinished stages' residuals (independent), taken
    outside the longest path LP; the hypothetical completion of request r
    replaces its stage's residual z by max(z - D_r, 0).
  * Eq. (6)-(7): Delta_task(r | H) = L_i(H) - L_i(H + {r}); J_admit sums it
    over the admitted requests in their greedy order, H being the task's
    earlier admitted requests.
  * Eq. (8)-(10): J_move, J_redo, J_revoke.
  * Eq. (11): V_reuse = beta sum_{a in R'} n_a mu l_a / B_swap, n_a counting
    the not-yet-started stages of agent a whose only unfinished predecessor
    is running.
  * Eq. (12)-(13): g_i = 1 + rho ln(1 + (t - tau_i) / H_age) scales the
    admission terms; Score = J_admit^age - J_move - J_redo - J_revoke + V_reuse.
  * GreedyPack (Sec. 4.5) and Alg. 1, then Eq. (14): the argmax with
    deterministic ties.

Readings where the paper is silent (beta, rho, H_age, M, K, tie order, the
exhausted-profile residual) are the ones the design notes list; the scenario
format is the plain dict of the workflow generator.
"""

from __future__ import annotations

import itertools
import math

from .movement import movement_cost, movement_time, resident_after

RTOL = 1e-9


# --------------------------------------------------------------------------- Eq. (4)-(6)

def residual(samples, served, status):
    """Eq. (4): the residual distribution of one stage as (value, prob) pairs."""
    if status == "done":
        return [(0.0, 1.0)]
    if served > 0:
        left = [x - served for x in samples if x > served]
        if not left:
            return [(0.0, 1.0)]
    else:
        left = list(samples)
    counts = {}
    for x in left:
        counts[float(x)] = counts.get(float(x), 0) + 1
    total = len(left)
    return [(x, c / total) for x, c in sorted(counts.items())]


def longest_path(edges, n, z):
    """LP(G, z): the heaviest path of the DAG with stage weights z."""
    succ = {v: [w for u, w in edges if u == v] for v in range(n)}
    memo = {}

    def down(v):
        if v not in memo:
            memo[v] = z[v] + max((down(w) for w in succ[v]), default=0.0)
        return memo[v]

    return max(down(v) for v in range(n))


def expected_remaining_path(sc, task, cut):
    """Eq. (5): E[LP] of a task, stage v's residual reduced by cut[v]."""
    n = len(sc["dag"]["agent"])
    dists = []
    for v in range(n):
        st = task["stages"][v]
        d = residual(sc["profiles"][v], float(st.get("served", 0.0)), st["status"])
        dists.append([(max(x - cut.get(v, 0.0), 0.0), p) for x, p in d])
    total = 0.0
    for combo in itertools.product(*dists):
        z = [x for x, _ in combo]
        prob = 1.0
        for _, p in combo:
            prob *= p
        total += prob * longest_path(sc["dag"]["edges"], n, z)
    return total


def task_progress(sc, task, stage, d_hat, earlier):
    """Eq. (6): Delta_task of a request of ``stage`` (expected service d_hat),
    given the task's earlier hypothetical completions ``earlier`` (a list of
    (stage, d_hat) pairs)."""
    before, after = {}, {}
    for v, x in earlier:
        before[v] = before.get(v, 0.0) + x
        after[v] = after.get(v, 0.0) + x
    after[stage] = after.get(stage, 0.0) + d_hat
    return expected_remaining_path(sc, task, before) - expected_remaining_path(sc, task, after)


# --------------------------------------------------------------------------- Eq. (8)-(13)

def age_weight(now, arrival, rho, h_age):
    """Eq. (12)."""
    return 1.0 + rho * math.log(1.0 + (now - arrival) / h_age)


def downstream_ready(sc):
    """n_a(t) of Eq. (11)."""
    agent = sc["dag"]["agent"]
    n = {}
    for t in sc["tasks"]:
        st = t["stages"]
        for w in range(len(agent)):
            if st[w]["status"] != "pending":
                continue
            preds = [u for u, v in sc["dag"]["edges"] if v == w]
            unfinished = [u for u in preds if st[u]["status"] != "done"]
            if len(unfinished) == 1 and st[unfinished[0]]["status"] == "running":
                n[agent[w]] = n.get(agent[w], 0) + 1
    return n


def score(sc, prm, resident_new, admitted_with_gain, preempted):
    """Eq. (13) of a candidate.  admitted_with_gain: (request, g * Delta) in
    the greedy order."""
    reqs = {r["id"]: r for r in sc["requests"]}
    agent = sc["dag"]["agent"]
    plen = {a: l for a, l in enumerate(sc["prefix_len"])}
    j_admit = sum(g for _, g in admitted_with_gain)
    adm = [(reqs[r]["task"], agent[reqs[r]["stage"]]) for r, _ in admitted_with_gain]
    j_move = movement_cost(prm.mu, prm.b_swap, plen, set(sc["resident"]), set(resident_new), adm)
    j_redo = sum(prm.t_decode * reqs[r].get("generated", 0) for r in preempted)
    j_revoke = sum(reqs[r].get("credit", 0.0) for r in preempted)
    n = downstream_ready(sc)
    v_reuse = prm.beta * sum(n.get(a, 0) * prm.mu * plen[a] / prm.b_swap for a in resident_new)
    return j_admit - j_move - j_redo - j_revoke + v_reuse


# --------------------------------------------------------------------------- GreedyPack and Alg. 1

def close(a, b):
    return abs(a - b) <= RTOL * max(1.0, abs(a), abs(b))


def greedy_pack(sc, prm, prefix_set):
    """GreedyPack(R): list of candidate states (dicts with resident, running,
    admitted, preempted, score)."""
    reqs = {r["id"]: r for r in sc["requests"]}
    tasks = {t["id"]: t for t in sc["tasks"]}
    agent = sc["dag"]["agent"]
    plen = sc["prefix_len"]
    a_of = lambda r: agent[reqs[r]["stage"]]
    running = sorted(r for r in reqs if reqs[r]["running"])
    waiting = sorted(r for r in reqs if not reqs[r]["running"])
    R = set(prefix_set)
    retained = [r for r in running if a_of(r) in R]
    preempted = [r for r in running if a_of(r) not in R]
    if prm.K and len(preempted) > prm.K:
        return []
    uncovered = R - {a_of(r) for r in retained}
    for a in uncovered:
        if not any(a_of(r) == a for r in waiting):
            return []
    reserve = {a: min(reqs[r]["d"] for r in waiting if a_of(r) == a) for a in uncovered}
    used = sum(plen[a] for a in R) + sum(reqs[r]["d"] for r in retained)
    if used + sum(reserve.values()) > prm.budget:
        return []
    if prm.K and len(uncovered) > prm.K:
        return []

    states = []
    admitted = []        # (request, g * Delta) in order
    history = {}         # task -> [(stage, d_hat)] of its admitted requests

    def emit():
        if uncovered:
            return
        states.append(dict(resident=sorted(R), running=sorted(retained + [r for r, _ in admitted]),
                           admitted=[r for r, _ in admitted], preempted=sorted(preempted),
                           score=score(sc, prm, R, admitted, preempted)))

    emit()
    remaining = [r for r in waiting if a_of(r) in R]
    while remaining:
        if prm.K and len(admitted) >= prm.K:
            break
        represented = {reqs[r]["task"] for r in retained} | {reqs[r]["task"] for r, _ in admitted}
        choice = None
        for r in remaining:
            q = reqs[r]
            others = [a for a in uncovered if a != a_of(r)]
            if used + q["d"] + sum(reserve[a] for a in others) > prm.budget:
                continue
            if prm.K and len(admitted) + 1 + len(others) > prm.K:
                continue
            task = tasks[q["task"]]
            delta = task_progress(sc, task, q["stage"], q["d_hat"], history.get(q["task"], []))
            g = age_weight(sc["now"], task["arrival"], prm.rho, prm.h_age)
            rate = g * delta / max(q["d"], 1.0)
            if choice is None:
                choice = (r, rate, g * delta)
                continue
            r0, rate0, _ = choice
            if close(rate, rate0):
                # equal rates: a represented task first, then the lower id
                rep, rep0 = q["task"] in represented, reqs[r0]["task"] in represented
                if (rep and not rep0) or (rep == rep0 and r < r0):
                    choice = (r, rate, g * delta)
            elif rate > rate0:
                choice = (r, rate, g * delta)
        if choice is None:
            break
        r, _, gain = choice
        q = reqs[r]
        remaining.remove(r)
        admitted.append((r, gain))
        history.setdefault(q["task"], []).append((q["stage"], q["d_hat"]))
        used += q["d"]
        uncovered.discard(a_of(r))
        emit()
    return states


def _tie_key(st, r_t):
    return (len(st["preempted"]), len(set(st["resident"]) ^ set(r_t)), tuple(st["resident"]), tuple(st["running"]))


def best_of(states, r_t):
    """Eq. (14): the highest score; equal scores go to fewer preemptions,
    fewer moved prefixes, then the smaller resident and running sets."""
    best = None
    for st in states:
        if best is None:
            best = st
        elif close(st["score"], best["score"]):
            if _tie_key(st, r_t) < _tie_key(best, r_t):
                best = st
        elif st["score"] > best["score"]:
            best = st
    return best


def phi(states):
    return max((s["score"] for s in states), default=-math.inf)


def repair(R, active):
    R = set(R)
    out = []
    for a in sorted(R):
        out.append(R - {a})
        for b in active:
            if b not in R:
                out.append((R - {a}) | {b})
    return out


def better_phi(new, old):
    return new > old and not close(new, old) if old != -math.inf else new > -math.inf


def hierarchical_search(sc, prm):
    """Alg. 1: the selected state (a dict as greedy_pack's)."""
    reqs = sc["requests"]
    agent = sc["dag"]["agent"]
    active = sorted({agent[r["stage"]] for r in reqs})
    r_t = set(sc["resident"])
    cands = []
    if len(active) <= prm.M:
        for k in range(len(active) + 1):
            for sub in itertools.combinations(active, k):
                cands += greedy_pack(sc, prm, sub)
    else:
        r_g = set(r_t)
        p_pair = False
        for R in [r_g] + repair(r_g, active):
            cands += greedy_pack(sc, prm, R)
        while True:
            base = phi(greedy_pack(sc, prm, r_g))
            best = None
            for a in active:
                if a in r_g:
                    continue
                sts = greedy_pack(sc, prm, r_g | {a})
                cands += sts
                if best is None or better_phi(phi(sts), best[0]):
                    best = (phi(sts), r_g | {a})
            if best is not None and better_phi(best[0], base):
                r_g = best[1]
            elif not p_pair:
                p_pair = True
                best = None
                rest = [a for a in active if a not in r_g]
                for a, b in itertools.combinations(rest, 2):
                    sts = greedy_pack(sc, prm, r_g | {a, b})
                    cands += sts
                    if best is None or better_phi(phi(sts), best[0]):
                        best = (phi(sts), r_g | {a, b})
                if best is not None and better_phi(best[0], base):
                    r_g = best[1]
                else:
                    break
            else:
                break
        for R in repair(r_g, active):
            cands += greedy_pack(sc, prm, R)
        running = sorted(r["id"] for r in reqs if r["running"])
        cands.append(dict(resident=sorted(r_t), running=running, admitted=[], preempted=[],
                          score=score(sc, prm, r_t, [], [])))
    incumbent_empty = not any(r["running"] for r in reqs)
    if incumbent_empty and any(c["running"] for c in cands):
        cands = [c for c in cands if c["running"]]
    return best_of(cands, r_t)


def feasible(sc, prm, running_ids):
    """Eq. (2) for the state whose running set is ``running_ids`` (its
    resident set being their agents): sum of l_a over R' plus sum of d_r."""
    reqs = {r["id"]: r for r in sc["requests"]}
    agent = sc["dag"]["agent"]
    resident = resident_after(agent[reqs[r]["stage"]] for r in running_ids)
    return sum(sc["prefix_len"][a] for a in resident) + sum(reqs[r]["d"] for r in running_ids) <= prm.budget
