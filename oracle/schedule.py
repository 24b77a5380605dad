"""Tail-batching round policy, simulated on forced lengths -- oracle, test infrastructure only.

Paper section 3 ("Tail Batching"): each rollout step needs P0 prompts with R0
responses each.  A short round launches ceil(eta_p*P0) prompts with
ceil(eta_r*R0) responses each (section 6.3 sets the two factors separately;
section 3 uses one eta for both) and keeps only the first P0 prompts to complete,
each with its first R0 responses to complete ("race to completion").  Prompts
aborted in a short round join a FIFO long-prompt queue; once the queue holds
P0 prompts they run as a long round with speculation disabled, so every
prompt is eventually scheduled and none is dropped.

Time is counted in decode steps: response r of prompt p, generated one token
per step, completes after L[p][r] steps.  A prompt completes when R0 of its
responses have.  Readings for cases the paper leaves open:
  * completion ties go to the lower prompt (or response) index;
  * the round ends when its P0-th prompt completes; every response still
    running then is aborted, and each accepted prompt's surplus responses
    stop as soon as that prompt completes;
  * when fewer than ceil(eta*P0) fresh prompts remain, the short round
    launches what is left and keeps min(P0, launched) of them;
  * when no fresh prompt remains, queued prompts are flushed in long rounds
    of up to P0 prompts;
  * a product eta*k within one part in 10^6 of an integer counts as that
    integer (eta = 1.1 and k = 10 launch 11, not 12).
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence


def spec_count(eta: float, k: int) -> int:
    """ceil(eta * k), reading products within 1e-6 relative of an integer as that integer."""
    x = eta * k
    return math.ceil(x - 1e-6 * x)


def _kth_smallest(vals: Sequence[int], k: int) -> int:
    return sorted(vals)[k - 1]


def _first_k(vals: Sequence[int], k: int) -> List[int]:
    """Indices of the k smallest values, lower index first on ties."""
    return sorted(range(len(vals)), key=lambda r: (vals[r], r))[:k]


def short_round(lens: Sequence[Sequence[int]], launched: List[int], P0: int, R0: int,
                eta_r: float) -> Dict:
    r_spec = spec_count(eta_r, R0)
    done_at = {p: _kth_smallest(lens[p][:r_spec], R0) for p in launched}
    keep_n = min(P0, len(launched))
    order = sorted(launched, key=lambda p: (done_at[p], p))
    accepted = sorted(order[:keep_n])
    rejected = sorted(order[keep_n:])
    t_round = max((done_at[p] for p in accepted), default=0)
    run = {}
    for p in launched:
        stop = done_at[p] if p in accepted else t_round
        for r in range(r_spec):
            run[(p, r)] = min(lens[p][r], stop)
    kept = {p: sorted(_first_k(lens[p][:r_spec], R0)) for p in accepted}
    return {"kind": "short", "launched": list(launched), "accepted": accepted,
            "rejected": rejected, "kept": kept, "time": t_round, "run": run}


def long_round(lens: Sequence[Sequence[int]], prompts: List[int], R0: int) -> Dict:
    run = {(p, r): lens[p][r] for p in prompts for r in range(R0)}
    return {"kind": "long", "launched": list(prompts), "accepted": list(prompts),
            "rejected": [], "kept": {p: list(range(R0)) for p in prompts},
            "time": max(run.values(), default=0), "run": run}


def plan_tail_batching(lens: Sequence[Sequence[int]], P0: int, R0: int, eta: float,
                       eta_r: Optional[float] = None) -> List[Dict]:
    """Rounds for prompts 0..n-1 submitted in order; lens[p] holds >= ceil(eta_r*R0) lengths.
    eta is the prompt factor eta_p and, unless eta_r is given, the response factor too."""
    eta_r = eta if eta_r is None else eta_r
    p_spec = spec_count(eta, P0)
    fresh = list(range(len(lens)))
    queue: List[int] = []
    rounds = []
    while fresh or queue:
        if len(queue) >= P0 or (not fresh and queue):
            take, queue = queue[:P0], queue[P0:]
            rounds.append(long_round(lens, take, R0))
            continue
        launched, fresh = fresh[:p_spec], fresh[p_spec:]
        rnd = short_round(lens, launched, P0, R0, eta_r)
        queue.extend(rnd["rejected"])
        rounds.append(rnd)
    return rounds


def plan_unscheduled(lens: Sequence[Sequence[int]], P0: int, R0: int) -> List[Dict]:
    """Baseline: consecutive batches of P0 prompts x R0 responses, no speculation."""
    n = len(lens)
    return [long_round(lens, list(range(s, min(n, s + P0))), R0) for s in range(0, n, P0)]


def slot_idle(run_steps: Sequence[int], t_round: int) -> float:
    """Fraction of sequence-slot time spent waiting for the round's end."""
    if not run_steps or t_round == 0:
        return 0.0
    return sum(t_round - t for t in run_steps) / (len(run_steps) * t_round)
