"""Prefix-movement cost of a residency transition.

TEST INFRASTRUCTURE ONLY: imported by tests, never by the product path.

Sec. 3 ("Joint prefix-request state"): the GPU state is the set R of
resident agent prefixes and the set Q of running requests; a request can run
only when its agent's prefix is resident, and idle prefixes are not kept, so
after a transition the resident set is exactly the agents of the running
requests.  Sec. 4.2 ("Prefix-movement delay", Eq. (8)): the prefixes leaving
(R_out = R_t minus R') and entering (R_in = R' minus R_t) the resident set are
moved one after another; with mu KV bytes per prefix token and a swap
bandwidth B_swap the transition takes mu / B_swap times the summed lengths of
both sets, and its cost J_move is that time times the number of distinct
admitted tasks that wait for an incoming prefix.
"""

from __future__ import annotations

from typing import Iterable, Mapping


def resident_after(request_agents: Iterable[int]) -> set:
    """Sec. 3: R' holds exactly the agents of the requests in Q'
    (requests without an agent, given as -1, hold no prefix)."""
    return {int(a) for a in request_agents if int(a) >= 0}


def transition_sets(r_before: Iterable[int], r_after: Iterable[int]):
    """(R_in, R_out) of Eq. (8): prefixes entering and leaving."""
    before, after = set(r_before), set(r_after)
    return after - before, before - after


def movement_time(mu: float, b_swap: float, prefix_len: Mapping[int, int], r_before, r_after) -> float:
    """Eq. (8): seconds for the transition's transfers, serialized."""
    r_in, r_out = transition_sets(r_before, r_after)
    tokens = sum(int(prefix_len[a]) for a in r_out) + sum(int(prefix_len[a]) for a in r_in)
    return mu / b_swap * tokens


def movement_cost(mu, b_swap, prefix_len, r_before, r_after, admitted) -> float:
    """Eq. (8): J_move = T_move times |T_in|, T_in being the distinct tasks
    of admitted requests whose agent's prefix is incoming.  ``admitted`` is a
    list of (task, agent) pairs, one per admitted request."""
    r_in, _ = transition_sets(r_before, r_after)
    waiting = {task for task, agent in admitted if agent in r_in}
    return movement_time(mu, b_swap, prefix_len, r_before, r_after) * len(waiting)
