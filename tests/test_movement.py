"""The prefix-movement oracle (Sec. 3 residency rule, Sec. 4.2 Eq. (8)) on
CPU, pinned by closed cases of the definition: no transition costs nothing,
evicting a prefix and loading it back costs two single transfers, costs add
over disjoint transitions, and J_move counts each waiting task once (a
hand-worked example)."""

import pytest

from oracle import movement as OM

MU = 4096.0          # bytes per prefix token: K and V, 8 KV heads, d = 128, bf16
B_SWAP = 50e9        # bytes per second


def test_resident_set_is_the_agents_of_running_requests():
    assert OM.resident_after([3, 1, 3, -1, 1]) == {1, 3}
    assert OM.resident_after([]) == set()


def test_no_transition_moves_nothing():
    lens = {0: 2048, 1: 700}
    assert OM.movement_time(MU, B_SWAP, lens, {0, 1}, {1, 0}) == 0.0
    assert OM.movement_cost(MU, B_SWAP, lens, {0, 1}, {0, 1}, [(7, 0), (8, 1)]) == 0.0


def test_single_load_and_round_trip():
    lens = {5: 1000}
    one = OM.movement_time(MU, B_SWAP, lens, set(), {5})
    assert one == pytest.approx(1000 * 4096 / 50e9)                   # 81.92 us
    assert OM.movement_time(MU, B_SWAP, lens, {5}, set()) == one      # eviction costs the same
    # out then back in: two transitions, twice the single transfer
    assert OM.movement_time(MU, B_SWAP, lens, {5}, set()) + one == pytest.approx(2 * one)


def test_swap_counts_both_directions_and_adds_over_disjoint_transitions():
    lens = {0: 512, 1: 8192, 2: 300, 3: 64}
    swap = OM.movement_time(MU, B_SWAP, lens, {0, 2}, {1, 2})      # 0 out, 1 in, 2 stays
    assert swap == pytest.approx((512 + 8192) * MU / B_SWAP)
    a = OM.movement_time(MU, B_SWAP, lens, {0}, {1})
    b = OM.movement_time(MU, B_SWAP, lens, {3}, {2})
    both = OM.movement_time(MU, B_SWAP, lens, {0, 3}, {1, 2})
    assert both == pytest.approx(a + b)


def test_cost_counts_each_waiting_task_once():
    # Hand example: agents 0 (resident, stays) and 1 (incoming, 100 tokens).
    # Admitted requests (task, agent): task 4 has two requests on agent 1,
    # task 5 one on agent 1, task 6 one on agent 0 (no wait).  T_in = {4, 5}.
    lens = {0: 50, 1: 100}
    t = 100 * MU / B_SWAP
    j = OM.movement_cost(MU, B_SWAP, lens, {0}, {0, 1}, [(4, 1), (4, 1), (5, 1), (6, 0)])
    assert j == pytest.approx(2 * t)


def test_paced_load_parts_keep_every_copy_in_order():
    """The copy-engine load cut into parts (one per event it waits for):
    every page copied once, in order, the parts as even as the page counts
    allow, and exactly as many parts as events."""
    from paper_2608_25523_amd.movement import Mover

    ops = [("k", "v", 0, 100, 10), ("k", "v", 50, 7, 3), ("k", "v", 200, 30, 20)]
    want = [(d0 + i, s0 + i) for (_, _, d0, s0, m) in ops for i in range(m)]
    for n in (1, 2, 4, 7, 33, 40):
        parts = Mover._split(ops, n)
        assert len(parts) == n
        flat = [(d0 + i, s0 + i) for p in parts for (_, _, d0, s0, m) in p for i in range(m)]
        assert flat == want
        sizes = [sum(op[4] for op in p) for p in parts]
        assert max(sizes) == -(-33 // n) or n > 33
    assert Mover._split([], 3) == [[], [], []]
