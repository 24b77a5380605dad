"""Tail batching executed on the engine (rp_rollout_tail_batched) on the GPU.

The online executor observes completions step by step and aborts responses;
its decisions must equal the planner's (native and oracle) on the same forced
lengths, every response's tokens must be a prefix of (or equal to) the same
sequence generated without scheduling, and every page must come back.  The
fp32 model is used because its kernels reduce each output in a fixed order
whatever the batch, so token streams do not depend on batch composition.
"""
import math

import numpy as np
import pytest

from oracle import schedule as osch
from tests.gpu_helpers import log, rp, to_device
from workloads import SHAPES, make_rl_batch, make_weights

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

DEV = torch.device("cuda:0")


@pytest.fixture(scope="module")
def tiny():
    s = SHAPES["tiny"]
    return s, to_device(make_weights(s, seed=0, device="cpu"), DEV)


def _engine(shape, wdev, max_seqs, pages, max_ctx=128):
    R = rp()
    return R.Engine(shape, R.weights_for_engine(wdev), max_seqs=max_seqs, max_prefill_tokens=512,
                    max_context=max_ctx, kv_pages=pages)


def _expected_lengths(plan_rounds, n, r_spec):
    """Tokens each response generated in the last round it ran in."""
    last = np.zeros((n, r_spec), np.int32)
    for rnd in plan_rounds:
        for (p, r), t in rnd["run"].items():
            if t > 0:
                last[p, r] = t
    return last


CASES = [  # n_prompts, P0, R0, eta_p, eta_r, seed
    (12, 4, 2, 1.5, 1.5, 11),
    (10, 3, 3, 1.25, 1.25, 12),
    (7, 2, 2, 1.0, 1.0, 13),
    (11, 3, 2, 1.0, 2.0, 14),     # responses only: no prompt is ever queued
    (13, 2, 3, 1.5, 1.0, 15),     # prompts only
]


@pytest.mark.parametrize("n_prompts,P0,R0,eta_p,eta_r,seed", CASES)
def test_online_tail_batching_matches_plan_and_unscheduled_tokens(tiny, n_prompts, P0, R0, eta_p, eta_r, seed):
    s, wd = tiny
    R = rp()
    r_spec = math.ceil(eta_r * R0)
    b = make_rl_batch(s, n_prompts, r_spec, p_lo=8, p_hi=40, median=24, sigma_p=0.7, sigma_r=0.5, lo=1, hi=80,
                      seed=seed, sample_seed=5, temperature=1.0)
    log(f"tail-batched tiny: prompts={n_prompts} P0={P0} R0={R0} eta_p={eta_p} eta_r={eta_r} seed={seed}")
    eng = _engine(s, wd, max_seqs=64, pages=128)
    resp, glen, acc, kept, stats = eng.rollout_tail_batched(b.seq_ids, b.prompt_tokens, b.prompt_offsets,
                                                            b.max_new, b.sample_seed, b.temperature, P0, R0, eta_p,
                                                            eta_r)
    plan = osch.plan_tail_batching(b.max_new.tolist(), P0, R0, eta_p, eta_r)
    nat, nat_acc, nat_kept = R.rp_plan_tail_batching(b.max_new, P0, R0, eta_p, eta_r)
    # decisions
    assert len(stats) == len(plan) == len(nat)
    for k, (st, rnd) in enumerate(zip(stats, plan)):
        assert st["round_id"] == k and st["kind"] == (rnd["kind"] == "long")
        assert st["decode_steps"] == rnd["time"] - 1, (k, st, rnd["time"])
        assert st["n_seqs"] == len(rnd["launched"]) * (r_spec if rnd["kind"] == "short" else R0)
        assert st["generated_tokens"] == sum(rnd["run"].values())
        for p in rnd["accepted"]:
            assert acc[p] == k
            assert sorted(np.flatnonzero(kept[p]).tolist()) == sorted(rnd["kept"][p])
    assert np.array_equal(acc, nat_acc) and np.array_equal(kept, nat_kept)
    assert np.array_equal(glen, _expected_lengths(plan, n_prompts, r_spec))
    # tokens: the same sequences generated with no scheduling, to full length
    u = b.sequences(range(n_prompts), r_spec)
    full, _ = eng.rollout(u.seq_ids, u.prompt_tokens, u.prompt_offsets, u.max_new, b.sample_seed, b.temperature)
    off = np.concatenate([[0], np.cumsum(b.max_new.reshape(-1))])
    for i in range(u.n):
        p, r = divmod(i, r_spec)
        g = glen[p, r]
        assert np.array_equal(resp[off[i]:off[i] + g], full[off[i]:off[i] + g]), (p, r, g)
        if kept[p, r]:
            assert g == b.max_new[p, r]
    # every slot and page came back: 64 sequences of 2 pages fill the 128-page pool
    ids = np.arange(10**6, 10**6 + 64, dtype=np.int64)
    eng.prefill(ids, np.tile(np.arange(8, dtype=np.int32), 64), np.arange(65, dtype=np.int64) * 8,
                np.full(64, 120, np.int32))
    eng.abort(ids)
    eng.close()


def test_no_speculation_equals_unscheduled_steps(tiny):
    """With eta = 1 every short round accepts every prompt: the rounds are the unscheduled steps."""
    s, wd = tiny
    P0, R0 = 3, 2
    b = make_rl_batch(s, 9, R0, p_lo=8, p_hi=40, median=24, sigma_p=0.7, sigma_r=0.5, lo=1, hi=80, seed=21)
    eng = _engine(s, wd, max_seqs=16, pages=64)
    resp, glen, acc, kept, stats = eng.rollout_tail_batched(b.seq_ids, b.prompt_tokens, b.prompt_offsets,
                                                            b.max_new, b.sample_seed, b.temperature, P0, R0, 1.0)
    u = b.sequences(range(9), R0)
    full, ust = eng.rollout(u.seq_ids, u.prompt_tokens, u.prompt_offsets, u.max_new, b.sample_seed, b.temperature,
                            (np.arange(u.n) // (P0 * R0)).astype(np.int32))
    eng.close()
    assert np.array_equal(resp, full)
    assert kept.all() and np.array_equal(glen, b.max_new) and acc.tolist() == [0, 0, 0, 1, 1, 1, 2, 2, 2]
    assert [st["kind"] for st in stats] == [0, 0, 0]
    assert [st["decode_steps"] for st in stats] == [st["decode_steps"] for st in ust]


def test_short_round_that_cannot_start_at_once_is_rejected(tiny):
    s, wd = tiny
    R = rp()
    b = make_rl_batch(s, 6, 3, p_lo=8, p_hi=40, median=24, sigma_p=0.7, sigma_r=0.5, lo=1, hi=80, seed=31)
    eng = _engine(s, wd, max_seqs=8, pages=64)     # a short round launches 3 prompts x 3 = 9 responses
    with pytest.raises(R.RollpackError) as e:
        eng.rollout_tail_batched(b.seq_ids, b.prompt_tokens, b.prompt_offsets, b.max_new, 0, 1.0, 2, 2, 1.5)
    assert e.value.status == 7
    # nothing ran and the engine is still usable
    resp, glen, acc, kept, stats = eng.rollout_tail_batched(b.seq_ids[:2, :2], b.prompt_tokens,
                                                            b.prompt_offsets[:3], b.max_new[:2, :2], 0, 1.0, 1, 2,
                                                            1.0)
    eng.close()
    assert kept.all() and len(stats) == 2


def test_step_trace_records_every_step(tiny):
    """rp_step_trace_*: one record per prefill chunk and decode step, with rows, context sums and round ids."""
    s, wd = tiny
    from workloads import make_workload
    wl = make_workload("tiny")
    mn = np.array([5, 64, 1, 30, 64, 2, 17, 40], np.int32)
    eng = _engine(s, wd, max_seqs=8, pages=32)
    eng.step_trace(1000)
    _, st = eng.rollout(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, mn, 3, 1.0,
                        np.array([4, 4, 4, 4, 9, 9, 9, 9], np.int32))
    rec = eng.step_trace_read()
    eng.step_trace(0)
    eng.close()
    dec = rec[rec["kind"] == 0]
    assert len(dec) == sum(x["decode_steps"] for x in st) and (rec["kind"] == 1).sum() == 2
    assert set(rec["round_id"].tolist()) == {4, 9} and (rec["ms"] > 0).all()
    # decode rows: live sequences per step of each round (all admitted together, one token per step)
    for rid, lens in ((4, mn[:4]), (9, mn[4:])):
        rows = dec[dec["round_id"] == rid]["rows"].tolist()
        assert rows == [int((lens > j).sum()) for j in range(1, int(lens.max()))]
        ctx = dec[dec["round_id"] == rid]["sum_ctx"].tolist()
        assert ctx == [int(sum(32 + j for L in lens if L > j)) for j in range(1, int(lens.max()))]
