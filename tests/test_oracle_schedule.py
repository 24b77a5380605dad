"""Pins of the tail-batching policy oracle (CPU only).

The sort-based planner is checked against an independent step-by-step
simulation of race-to-completion on small random cases, and against the
invariants the paper states (section 3): every prompt is eventually scheduled
exactly once, short rounds keep exactly P0 prompts with R0 responses each,
and long rounds (from the FIFO long-prompt queue) run without speculation.
"""
import math

import numpy as np
import pytest

from oracle import schedule as osch


def _simulate_short(lens, launched, P0, R0, eta):
    """Advance time one decode step at a time until P0 prompts have R0 finished responses."""
    r_spec = math.ceil(eta * R0)
    finished = {p: [] for p in launched}
    done = []
    keep_n = min(P0, len(launched))
    t = 0
    while len(done) < keep_n:
        t += 1
        newly = []
        for p in launched:
            if p in done:
                continue
            for r in range(r_spec):
                if lens[p][r] == t:
                    finished[p].append(r)
            if len(finished[p]) >= R0:
                newly.append(p)
        for p in sorted(newly):          # same-step completions: lower index first
            if len(done) < keep_n:
                done.append(p)
    # finished[p] is in finish order (by step, then response index): keep the first R0
    return sorted(done), t, {p: sorted(finished[p][:R0]) for p in done}


@pytest.mark.parametrize("seed", range(40))
def test_short_round_matches_step_simulation(seed):
    rng = np.random.default_rng(seed)
    P0, R0 = int(rng.integers(1, 5)), int(rng.integers(1, 4))
    eta_p, eta_r = (float(rng.choice([1.0, 1.25, 1.5, 2.0])) for _ in range(2))
    n = math.ceil(eta_p * P0)
    r_spec = math.ceil(eta_r * R0)
    lens = rng.integers(1, 12, size=(n, r_spec)).tolist()
    rnd = osch.short_round(lens, list(range(n)), P0, R0, eta_r)
    acc, t, kept = _simulate_short(lens, list(range(n)), P0, R0, eta_r)
    assert rnd["accepted"] == acc and rnd["time"] == t
    # kept responses: the first R0 to finish, lower index first among same-step finishes
    for p in acc:
        assert rnd["kept"][p] == kept[p]


@pytest.mark.parametrize("seed", range(20))
def test_plan_invariants(seed):
    rng = np.random.default_rng(100 + seed)
    P0, R0 = int(rng.integers(1, 6)), int(rng.integers(1, 5))
    eta_p, eta_r = [(1.25, 1.25), (1.0, 1.5), (1.5, 1.0), (1.25, 2.0)][seed % 4]
    n = int(rng.integers(1, 40))
    r_spec = math.ceil(eta_r * R0)
    lens = np.clip(np.rint(50 * np.exp(rng.standard_normal((n, r_spec)))), 1, 2000).astype(int).tolist()
    rounds = osch.plan_tail_batching(lens, P0, R0, eta_p, eta_r)
    seen = []
    queue_order = []
    for rnd in rounds:
        seen += rnd["accepted"]
        if rnd["kind"] == "long":
            assert rnd["launched"] == rnd["accepted"] and len(rnd["accepted"]) <= P0
            assert all(rnd["kept"][p] == list(range(R0)) for p in rnd["accepted"])
            assert all(rnd["run"][(p, r)] == lens[p][r] for p in rnd["accepted"] for r in range(R0))
            # FIFO: long rounds take the oldest queued prompts
            assert rnd["accepted"] == queue_order[:len(rnd["accepted"])]
            queue_order = queue_order[len(rnd["accepted"]):]
        else:
            assert len(rnd["launched"]) <= math.ceil(eta_p * P0)
            assert len(rnd["accepted"]) == min(P0, len(rnd["launched"]))
            assert all(len(rnd["kept"][p]) == R0 for p in rnd["accepted"])
            assert all(t <= rnd["time"] for t in rnd["run"].values())
            queue_order += rnd["rejected"]
    assert sorted(seen) == list(range(n))            # every prompt exactly once


def test_speculation_counts_read_decimal_factors():
    assert osch.spec_count(1.25, 128) == 160 and osch.spec_count(1.25, 8) == 10
    assert osch.spec_count(1.1, 10) == 11 and osch.spec_count(float(np.float32(1.1)), 10) == 11
    assert osch.spec_count(1.0, 7) == 7 and osch.spec_count(1.01, 10) == 11


def test_factor_one_on_both_sides_is_the_unscheduled_plan():
    """With eta_p = eta_r = 1 nothing is speculative: each round is one unscheduled step."""
    rng = np.random.default_rng(5)
    lens = rng.integers(1, 100, size=(12, 3)).tolist()
    tb = osch.plan_tail_batching(lens, 4, 3, 1.0)
    un = osch.plan_unscheduled(lens, 4, 3)
    assert [r["time"] for r in tb] == [r["time"] for r in un]
    assert [r["accepted"] for r in tb] == [r["accepted"] for r in un]


def test_response_only_speculation_never_queues():
    """eta_p = 1 launches exactly P0 prompts, all accepted: no prompt reaches the long queue (section 6.3)."""
    rng = np.random.default_rng(6)
    lens = rng.integers(1, 500, size=(20, 6)).tolist()
    rounds = osch.plan_tail_batching(lens, 5, 4, 1.0, 1.5)
    assert all(r["kind"] == "short" and not r["rejected"] for r in rounds)
    # each round ends when its slowest prompt has its 4 shortest of 6 responses
    for r in rounds:
        assert r["time"] == max(sorted(lens[p])[3] for p in r["launched"])


def test_unscheduled_and_slot_idle():
    lens = [[3, 9], [4, 4], [10, 1]]
    rounds = osch.plan_unscheduled(lens, 2, 2)
    assert [r["time"] for r in rounds] == [9, 10]
    assert osch.slot_idle([3, 9, 4, 4], 9) == pytest.approx((6 + 0 + 5 + 5) / 36)
    assert osch.slot_idle([], 5) == 0.0


def test_long_tail_moves_to_long_round():
    # prompt 2 only has long responses: it is aborted, queued and run in a long round
    lens = [[5, 6, 7], [4, 5, 6], [90, 95, 99], [6, 6, 6], [5, 5, 5]]
    rounds = osch.plan_tail_batching(lens, 2, 2, 1.5)
    assert rounds[0]["kind"] == "short" and 2 in rounds[0]["rejected"]
    longs = [r for r in rounds if r["kind"] == "long"]
    assert any(2 in r["accepted"] for r in longs)
