"""Seeded synthetic scheduling scenarios: a workflow DAG, tasks in flight,
their requests and the service profiles, as one plain dict.

This module only draws structure and numbers.  It holds none of the
scheduler's arithmetic, so both the scheduler and its plain reference read
what it produces.

Scenario format
  dag         {"agent": [agent of stage v], "edges": [[u, v], ...]} (u before v)
  prefix_len  [l_a]: static prefix tokens of agent a (Sec. 3)
  profiles    [[x, ...]]: per stage, observed total LLM service of that
              agent-stage pair in seconds (a point mass is one sample)
  tasks       [{"id", "arrival", "stages": [{"status", "served"}]}], status
              one of "pending" (not ready), "ready" (waiting, not started),
              "running" (started, not finished), "done"; served = e_{i,v}
  requests    [{"id", "task", "stage", "d" (KV tokens it reserves),
              "d_hat" (expected service, s), "running", "generated" (tokens
              to rebuild if preempted), "credit" (lambda_r if running)}]
  resident    [agents whose prefixes are resident] (R_t)
  now         the event time t

The paper's workloads (Sec. 5.1: Chain-3, DAG-4, DAG-10-Wide synthetic
workflows and MetaGPT traces) are not available; these stand-ins have the
same shapes of workflow.
"""

from __future__ import annotations

import copy

import numpy as np


def chain(n_stages: int):
    """A -> B -> C ...: stage v run by agent v."""
    return {"agent": list(range(n_stages)), "edges": [[v, v + 1] for v in range(n_stages - 1)]}


def fork_join(width: int):
    """Source -> `width` parallel stages -> sink; every stage its own agent."""
    edges = [[0, 1 + i] for i in range(width)] + [[1 + i, width + 1] for i in range(width)]
    return {"agent": list(range(width + 2)), "edges": edges}


DAGS = {
    "chain3": lambda: chain(3),
    "dag4": lambda: {"agent": [0, 1, 2, 3], "edges": [[0, 1], [0, 2], [1, 3], [2, 3]]},
    "wide10": lambda: fork_join(8),
}


def _ready(dag, status, v):
    preds = [u for u, w in dag["edges"] if w == v]
    return all(status[u] == "done" for u in preds)


def random_scenario(seed: int, dag: str = "chain3", n_tasks: int = 6, budget: float | None = None,
                    samples: int = 3, max_requests_per_stage: int = 2):
    """A seeded snapshot of tasks flowing through one DAG: each task has
    finished a random prefix of a topological order, its ready stages hold
    waiting requests, and some requests are running (their agents resident,
    within the budget).  Returns (scenario, budget)."""
    rng = np.random.default_rng(seed)
    g = DAGS[dag]()
    n = len(g["agent"])
    n_agents = max(g["agent"]) + 1
    plen = [int(x) for x in rng.integers(200, 2000, size=n_agents)]
    profiles = [sorted(float(x) for x in np.round(rng.uniform(0.5, 6.0, size=samples), 2)) for _ in range(n)]
    topo = list(range(n))            # stage ids are already in a topological order
    tasks, requests = [], []
    rid = 0
    for t in range(n_tasks):
        done_upto = int(rng.integers(0, n))
        status = ["done" if v < done_upto else "pending" for v in topo]
        for v in topo:
            if status[v] == "pending" and _ready(g, status, v):
                status[v] = "ready"
        stages = []
        for v in range(n):
            stages.append({"status": status[v], "served": 0.0})
        for v in range(n):
            if status[v] != "ready":
                continue
            if rng.random() < 0.3:       # a later ReAct round: some service already recorded
                stages[v]["served"] = float(np.round(rng.uniform(0.1, 2.0), 2))
                stages[v]["status"] = "running"
            for _ in range(int(rng.integers(1, max_requests_per_stage + 1))):
                requests.append({"id": rid, "task": t, "stage": v, "d": int(rng.integers(50, 600)),
                                 "d_hat": float(np.round(rng.uniform(0.3, 3.0), 2)), "running": False,
                                 "generated": 0, "credit": 0.0})
                rid += 1
        tasks.append({"id": t, "arrival": float(np.round(rng.uniform(0.0, 20.0), 2)), "stages": stages})
    budget = float(budget if budget is not None else int(rng.integers(1500, 5000)))
    # Some requests are already running: pick agents and requests that fit.
    resident, used = set(), 0.0
    for r in rng.permutation(len(requests)):
        q = requests[int(r)]
        a = g["agent"][q["stage"]]
        extra = q["d"] + (0 if a in resident else plen[a])
        if rng.random() < 0.4 and used + extra <= budget:
            q["running"] = True
            q["generated"] = int(rng.integers(0, 200))
            q["credit"] = float(np.round(rng.uniform(0.0, 2.0), 3))
            tasks[q["task"]]["stages"][q["stage"]]["status"] = "running"
            resident.add(a)
            used += extra
    # A running stage's task: its pending successors may be about to become ready.
    return {"dag": g, "prefix_len": plen, "profiles": profiles, "tasks": tasks, "requests": requests,
            "resident": sorted(resident), "now": float(np.round(rng.uniform(20.0, 40.0), 2))}, budget


def permuted(scenario, seed: int):
    """The same scenario with its request and task lists in another order
    (ids unchanged)."""
    rng = np.random.default_rng(seed)
    sc = copy.deepcopy(scenario)
    sc["requests"] = [sc["requests"][int(i)] for i in rng.permutation(len(sc["requests"]))]
    sc["tasks"] = [sc["tasks"][int(i)] for i in rng.permutation(len(sc["tasks"]))]
    return sc
