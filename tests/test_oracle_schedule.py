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
    return sorted(done), t, {p: sorted(finished[p])[:R0] for p in done}


@pytest.mark.parametrize("seed", range(40))
def test_short_round_matches_step_simulation(seed):
    rng = np.random.default_rng(seed)
    P0, R0 = int(rng.integers(1, 5)), int(rng.integers(1, 4))
    eta = float(rng.choice([1.0, 1.25, 1.5, 2.0]))
    n = math.ceil(eta * P0)
    r_spec = math.ceil(eta * R0)
    lens = rng.integers(1, 12, size=(n, r_spec)).tolist()
    rnd = osch.short_round(lens, list(range(n)), P0, R0, eta)
    acc, t, kept = _simulate_short(lens, list(range(n)), P0, R0, eta)
    assert rnd["accepted"] == acc and rnd["time"] == t
    # kept responses: any R0 finished by the prompt's completion step are valid;
    # the planner keeps the shortest with lower index first on ties
    for p in acc:
        assert sorted(lens[p][r] for r in rnd["kept"][p]) == sorted(lens[p][r] for r in kept[p])


@pytest.mark.parametrize("seed", range(20))
def test_plan_invariants(seed):
    rng = np.random.default_rng(100 + seed)
    P0, R0, eta = int(rng.integers(1, 6)), int(rng.integers(1, 5)), 1.25
    n = int(rng.integers(1, 40))
    r_spec = math.ceil(eta * R0)
    lens = np.clip(np.rint(50 * np.exp(rng.standard_normal((n, r_spec)))), 1, 2000).astype(int).tolist()
    rounds = osch.plan_tail_batching(lens, P0, R0, eta)
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
            assert len(rnd["accepted"]) == min(P0, len(rnd["launched"]))
            assert all(len(rnd["kept"][p]) == R0 for p in rnd["accepted"])
            assert all(t <= rnd["time"] for t in rnd["run"].values())
            queue_order += rnd["rejected"]
    assert sorted(seen) == list(range(n))            # every prompt exactly once


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
