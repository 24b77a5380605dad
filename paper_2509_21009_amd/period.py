"""One period of tail-batched RL steps against the same steps run unscheduled, on one GPU.

Each RL step needs P0 prompts with R0 responses (section 3).  Unscheduled, a
step runs its P0 x R0 responses to completion, so it lasts as long as its
longest response.  Tail batching runs the same prompts as short rounds that
launch ceil(eta_p*P0) prompts x ceil(eta_r*R0) responses and stop when P0
prompts have R0 finished responses, plus long rounds for the prompts those
rounds aborted (rp_rollout_tail_batched).  With eta_p = eta_r = 1.25 and
5 x P0 prompts, the queue reaches P0 after the fourth short round, so the
period is 4 short + 1 long round against 5 unscheduled steps.  Section 6.3's
sensitivity study varies eta_p and eta_r separately (--eta-p, --eta-r); the
prompt set stays the same, so times compare per RL step (P0 prompts).

Response lengths are forced and prompt-correlated (log L = log median +
sigma_p z_p + sigma_r z_pr), so hard prompts give long responses across the
board.  Weights are random at the named model's shape.  Prints one JSON line;
progress goes to stderr.  From the repository root:

    python3 -u paper_2509_21009_amd/period.py --model qwen2.5-0.5b --p0 128 --r0 8 --eta-p 1.25 --eta-r 1.25
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))


def log(msg: str):
    print(f"[period] {msg}", file=sys.stderr, flush=True)


def pages_for(tokens) -> np.ndarray:
    return (np.asarray(tokens, np.int64) + 63) // 64


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--model", default="qwen2.5-0.5b")
    ap.add_argument("--p0", type=int, default=128)
    ap.add_argument("--r0", type=int, default=8)
    ap.add_argument("--eta-p", type=float, default=1.25, help="prompt speculation factor")
    ap.add_argument("--eta-r", type=float, default=1.25, help="response speculation factor")
    ap.add_argument("--rl-steps", type=int, default=5, help="prompts = rl_steps x P0")
    ap.add_argument("--no-unscheduled", action="store_true", help="skip the unscheduled steps")
    ap.add_argument("--median", type=float, default=512.0)
    ap.add_argument("--sigma-p", type=float, default=0.6)
    ap.add_argument("--sigma-r", type=float, default=0.53)
    ap.add_argument("--len-lo", type=int, default=32)
    ap.add_argument("--len-hi", type=int, default=4096)
    ap.add_argument("--prompt-lo", type=int, default=64)
    ap.add_argument("--prompt-hi", type=int, default=512)
    ap.add_argument("--seed", type=int, default=106)
    args = ap.parse_args()

    import torch

    from paper_2509_21009_amd import rollpack as rp
    from workloads import SHAPES, make_rl_batch, make_weights

    rp.load_library()
    dev = torch.device("cuda:0")
    shape = SHAPES[args.model]
    P0, R0, eta_p, eta_r = args.p0, args.r0, args.eta_p, args.eta_r
    p_spec = math.ceil(eta_p * P0 * (1 - 1e-6))
    r_spec = math.ceil(eta_r * R0 * (1 - 1e-6))
    n_prompts = args.rl_steps * P0
    batch = make_rl_batch(shape, n_prompts, r_spec, p_lo=args.prompt_lo, p_hi=args.prompt_hi, median=args.median,
                          sigma_p=args.sigma_p, sigma_r=args.sigma_r, lo=args.len_lo, hi=args.len_hi,
                          seed=args.seed, sample_seed=args.seed + 100, name=f"{args.model}-rl")
    plen = np.diff(batch.prompt_offsets)
    need = pages_for(plen[:, None] + batch.max_new - 1)
    # pool: every round of the plan, and every unscheduled step, starts all of its responses at once
    plan, _, _ = rp.rp_plan_tail_batching(batch.max_new, P0, R0, eta_p, eta_r)
    round_pages = [int(need[r["launched"], :(r_spec if r["kind"] == "short" else R0)].sum()) for r in plan]
    step_pages = [int(need[i:i + P0, :R0].sum()) for i in range(0, n_prompts, P0)]
    kv_pages = max(round_pages + step_pages) + 64
    max_seqs = max(p_spec * r_spec, P0 * R0)
    log(f"{shape.name}: {n_prompts} prompts x {r_spec} responses, P0={P0} R0={R0} eta_p={eta_p} eta_r={eta_r}; "
        f"max_seqs={max_seqs} kv_pages={kv_pages}")
    weights = make_weights(shape, seed=0, device=dev)
    eng = rp.Engine(shape, rp.weights_for_engine(weights), max_seqs=max_seqs, max_prefill_tokens=32768,
                    max_context=int(plen.max() + batch.max_new.max()), kv_pages=kv_pages)

    # warm-up: kernels and allocator paths of both schedules on a few sequences
    w = batch.sequences(range(2), 2)
    eng.rollout(w.seq_ids, w.prompt_tokens, w.prompt_offsets, np.minimum(w.max_new, 16), batch.sample_seed,
                batch.temperature)
    torch.cuda.synchronize()

    log("tail-batched period")
    t0 = time.perf_counter()
    _, _, acc, kept, tb = eng.rollout_tail_batched(batch.seq_ids, batch.prompt_tokens, batch.prompt_offsets,
                                                   batch.max_new, batch.sample_seed, batch.temperature, P0, R0,
                                                   eta_p, eta_r)
    t_tb = time.perf_counter() - t0
    for s in tb:
        log(f"  round {s['round_id']} {'long' if s['kind'] else 'short'}: {s['n_seqs']} seqs, "
            f"{s['decode_steps']} steps, {s['makespan_ms'] / 1e3:.2f} s")

    n_steps = args.rl_steps
    us, t_un = [], 0.0
    if not args.no_unscheduled:
        log(f"unscheduled: {n_steps} steps of {P0} x {R0}")
        u = batch.sequences(range(n_steps * P0), R0)
        rid = (np.arange(u.n) // (P0 * R0)).astype(np.int32)
        t0 = time.perf_counter()
        _, us = eng.rollout(u.seq_ids, u.prompt_tokens, u.prompt_offsets, u.max_new, batch.sample_seed,
                            batch.temperature, rid)
        t_un = time.perf_counter() - t0
    for s in us:
        log(f"  step {s['round_id']}: {s['n_seqs']} seqs, {s['decode_steps']} steps, {s['makespan_ms'] / 1e3:.2f} s")
    eng.close()

    kept_tokens = int(batch.max_new[kept].sum())
    tb_tokens = int(sum(s["generated_tokens"] for s in tb))
    un_tokens = int(sum(s["generated_tokens"] for s in us))
    tb_s = sum(s["makespan_ms"] for s in tb) / 1e3
    un_s = sum(s["makespan_ms"] for s in us) / 1e3

    def rounds(stats):
        return [{"kind": ("long" if s["kind"] else "short") if stats is tb else "step", "seqs": s["n_seqs"],
                 "decode_steps": s["decode_steps"], "makespan_s": round(s["makespan_ms"] / 1e3, 3),
                 "prefill_s": round(s["prefill_ms"] / 1e3, 3),
                 "generated_tokens": s["generated_tokens"], "idle_slot_s": round(s["idle_slot_s"], 1),
                 "slot_idle": round(s["slot_idle"], 4)} for s in stats]

    out = {
        "metric": "RL-step rollout time over one tail-batching period vs unscheduled steps",
        "model": shape.name, "P0": P0, "R0": R0, "eta_p": eta_p, "eta_r": eta_r, "prompts": n_prompts,
        "rl_steps": n_steps,
        "lengths": f"prompt-correlated LogN(median {args.median:g}, sigma_p {args.sigma_p}, sigma_r "
                   f"{args.sigma_r}) in [{args.len_lo}, {args.len_hi}], prompts U[{args.prompt_lo}, "
                   f"{args.prompt_hi}], forced, T={batch.temperature}, synthetic",
        "tail_batched_s": round(tb_s, 3), "unscheduled_s": round(un_s, 3) if us else None,
        "tail_batched_s_per_rl_step": round(tb_s / n_steps, 3),
        "unscheduled_s_per_rl_step": round(un_s / n_steps, 3) if us else None,
        "speedup": round(un_s / tb_s, 3) if us and tb_s > 0 else None,
        "tail_batched_wall_s": round(t_tb, 3), "unscheduled_wall_s": round(t_un, 3),
        "tail_batched_generated_tokens": tb_tokens, "unscheduled_generated_tokens": un_tokens if us else None,
        "tail_batched_kept_tokens": kept_tokens,
        "tail_batched_idle_slot_s": round(sum(s["idle_slot_s"] for s in tb), 1),
        "unscheduled_idle_slot_s": round(sum(s["idle_slot_s"] for s in us), 1) if us else None,
        "tail_batched_rounds": rounds(tb), "unscheduled_steps": rounds(us),
        "accept_round_hist": np.bincount(acc, minlength=len(tb)).tolist(),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
