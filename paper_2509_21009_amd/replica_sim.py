"""Data-parallel rollout replicas, simulated from a measured step-time model (host only).

The paper's rollout runs many data-parallel replicas; each RL step waits for
the slowest one, which leaves the others idle (section 2.2).  Its stream
trainer (section 4.4, Algorithm 1) watches the fraction of completed
requests and, between 20% and 50% of them, at most once per 5% of new
completions, tries to hand half of the rollout GPUs to training: the running
requests of the freed replicas migrate to the others by recomputing their KV
from their tokens, provided the projected KV footprint of the survivors fits
their memory.  One GPU runs one replica here, so this module replays D
replicas on a clock driven by a step-time model fitted to the engine's own
per-step trace (rp_step_trace_*): a decode step over B rows with context sum
S takes c0 + c1 B + c2 S milliseconds; a prefill chunk of T tokens attending
to K keys in total takes d0 + d1 T + d2 K.

Readings where the paper is silent: requests are dealt to replicas in turn;
each replica admits all of its requests at once; the freed half is the half
with the fewest running requests; a migrated request is re-prefilled (prompt
and generated tokens) on the survivor with the fewest running requests; the
projected length of a running request is the mean of the historical lengths
above what it has already generated.

    python3 paper_2509_21009_amd/replica_sim.py --trace results/step_trace_7b.json
    python3 paper_2509_21009_amd/replica_sim.py --model 3.5135,0.018858,5.9101e-6 --prefill-model 0,0.013172,0
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import math
import os
import sys
from typing import Dict, List, Optional, Sequence

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))


@dataclasses.dataclass
class StepModel:
    decode: Sequence[float]   # c0, c1 (per row), c2 (per context token), ms
    prefill: Sequence[float]  # d0, d1 (per token), d2 (per attended key), ms

    def decode_ms(self, rows: int, sum_ctx: float) -> float:
        c0, c1, c2 = self.decode
        return c0 + c1 * rows + c2 * sum_ctx

    def prefill_ms(self, tokens: int, keys: float) -> float:
        d0, d1, d2 = self.prefill
        return d0 + d1 * tokens + d2 * keys

    @staticmethod
    def fit(records: np.ndarray) -> "StepModel":
        """Least squares over trace records [kind, round, rows, sum_ctx, ms]."""
        rec = np.asarray(records, np.float64)

        def ls(sel):
            r = rec[sel]
            if len(r) < 6:  # too few for three coefficients: a per-row (per-token) rate alone
                return [0.0, float(r[:, 4].sum() / max(r[:, 2].sum(), 1.0)), 0.0]
            A = np.stack([np.ones(len(r)), r[:, 2], r[:, 3]], axis=1)
            return np.linalg.lstsq(A, r[:, 4], rcond=None)[0].tolist()

        return StepModel(ls(rec[:, 0] == 0), ls(rec[:, 0] == 1))


@dataclasses.dataclass
class Req:
    idx: int
    prompt: int
    length: int        # tokens to generate (the first comes from the prefill)
    done: int = 0      # tokens generated so far
    finish_ms: float = math.nan


class Replica:
    """Continuous batching of its requests: one prefill, then decode steps until all are done."""

    def __init__(self, rid: int, reqs: List[Req], model: StepModel, max_prefill: int):
        self.rid, self.model, self.max_prefill = rid, model, max_prefill
        self.running: List[Req] = []
        self.clock = 0.0
        self.admit(reqs, recompute=False)

    def admit(self, reqs: List[Req], recompute: bool):
        """Prefill reqs (their prompts, or prompt + generated tokens when recomputing) in chunks."""
        toks = [r.prompt + (r.done if recompute else 0) for r in reqs]
        i = 0
        while i < len(reqs):
            t = keys = 0
            while i < len(reqs) and (t == 0 or t + toks[i] <= self.max_prefill):
                t += toks[i]
                keys += toks[i] * (toks[i] + 1) / 2
                i += 1
            self.clock += self.model.prefill_ms(t, keys)
        for r in reqs:
            if not recompute:
                r.done = 1
            else:
                r.done += 1  # the recompute prefill samples the next token
            if r.done >= r.length:
                r.finish_ms = self.clock
            else:
                self.running.append(r)

    def step(self) -> List[Req]:
        """One decode step; returns the requests it finished."""
        if not self.running:
            return []
        sum_ctx = sum(r.prompt + r.done for r in self.running)
        self.clock += self.model.decode_ms(len(self.running), sum_ctx)
        fin = []
        for r in self.running:
            r.done += 1
            if r.done >= r.length:
                r.finish_ms = self.clock
                fin.append(r)
        self.running = [r for r in self.running if r.done < r.length]
        return fin


def deal(n: int, replicas: int) -> List[List[int]]:
    return [list(range(r, n, replicas)) for r in range(replicas)]


def simulate(prompt: Sequence[int], length: Sequence[int], replicas: int, model: StepModel,
             max_prefill: int = 16384, trainer: Optional[Dict] = None) -> Dict:
    """Run one RL step's requests on `replicas` replicas; with `trainer`, apply Algorithm 1's scale-down.

    trainer: {"history": lengths of an earlier step, "kv_bytes_per_token": B, "kv_capacity": bytes per
    replica, "lo": 0.2, "hi": 0.5, "delta": 0.05}.
    """
    reqs = [Req(i, int(p), int(l)) for i, (p, l) in enumerate(zip(prompt, length))]
    reps = [Replica(r, [reqs[i] for i in ids], model, max_prefill) for r, ids in enumerate(deal(len(reqs), replicas))]
    active = list(reps)
    n = len(reqs)
    comp = sum(1 for r in reqs if r.done >= r.length)
    delta = comp
    scaled = None
    checks = []
    hist = np.sort(np.asarray(trainer["history"], np.float64)) if trainer else None

    def projected(r: Req) -> float:
        above = hist[hist > r.done]
        return float(above.mean()) if len(above) else float(max(r.done + 1, hist[-1]))

    while any(rep.running for rep in active):
        # advance the replica whose next step ends first (each replica steps on its own clock)
        rep = min((x for x in active if x.running), key=lambda x: x.clock)
        fin = rep.step()
        comp += len(fin)
        delta += len(fin)
        if trainer and scaled is None and fin:
            frac = comp / n
            if trainer["lo"] <= frac <= trainer["hi"] and delta / n >= trainer["delta"]:
                delta = 0
                now = rep.clock
                keep_n = len(active) - len(active) // 2
                order = sorted(active, key=lambda x: len(x.running))
                free, keep = order[:len(active) // 2], order[len(active) // 2:]
                moved = [r for x in free for r in x.running]
                load = {x.rid: list(x.running) for x in keep}
                for r in sorted(moved, key=lambda r: -r.done):
                    tgt = min(keep, key=lambda x: len(load[x.rid]))
                    load[tgt.rid].append(r)
                peak = max(sum((r.prompt + projected(r)) * trainer["kv_bytes_per_token"] for r in load[x.rid])
                           for x in keep) if keep else math.inf
                ok = bool(free) and keep_n > 0 and peak <= trainer["kv_capacity"]
                checks.append({"completed": round(frac, 4), "time_ms": round(now, 1), "free": len(free),
                               "migrated": len(moved), "projected_peak_gb": round(peak / 1e9, 2), "scaled": ok})
                if ok:
                    for x in keep:
                        x.clock = max(x.clock, now)
                    for x in free:
                        x.running = []
                        x.clock = now
                    for x in keep:
                        mine = [r for r in load[x.rid] if r not in x.running]
                        if mine:
                            x.admit(mine, recompute=True)
                    active = keep
                    scaled = {"time_ms": now, "completed": frac, "freed": len(free), "migrated": len(moved)}
    ends = [rep.clock for rep in reps]
    T = max(ends)
    out = {"replicas": replicas, "requests": n, "step_ms": T, "replica_end_ms": ends,
           "idle_gpu_s": sum(T - e for e in ends) / 1e3 if not scaled else None,
           "replica_idle_frac": sum(T - e for e in ends) / (replicas * T) if T > 0 else 0.0}
    if trainer:
        out["checks"] = checks
        out["scaled"] = scaled
        if scaled:
            out["train_gpu_s"] = scaled["freed"] * (T - scaled["time_ms"]) / 1e3
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--trace", default=None, help="JSON written by bench.py --step-trace")
    ap.add_argument("--model", default=None, help="decode step model c0,c1,c2 (ms) instead of a trace")
    ap.add_argument("--prefill-model", default="0,0,0", help="prefill chunk model d0,d1,d2 (ms) with --model")
    ap.add_argument("--replicas", type=int, default=16)
    ap.add_argument("--p0", type=int, default=128)
    ap.add_argument("--r0", type=int, default=8)
    ap.add_argument("--median", type=float, default=1024)
    ap.add_argument("--sigma-p", type=float, default=0.7)
    ap.add_argument("--sigma-r", type=float, default=0.6)
    ap.add_argument("--len-hi", type=int, default=16384)
    ap.add_argument("--kv-gb", type=float, default=250.0, help="KV memory per replica after weights")
    ap.add_argument("--seed", type=int, default=301)
    args = ap.parse_args()

    from workloads import SHAPES, make_rl_batch
    if args.trace:
        tr = json.load(open(args.trace))
        model = StepModel.fit(np.asarray(tr["records"]))
        n_rec = len(tr["records"])
    elif args.model:
        model = StepModel([float(x) for x in args.model.split(",")], [float(x) for x in args.prefill_model.split(",")])
        n_rec = 0
    else:
        ap.error("give --trace or --model")
    shape = SHAPES["qwen2.5-7b"]
    kvb = shape.layers * 2 * shape.n_kv * shape.head_dim * 2
    common = dict(p_lo=128, p_hi=1024, median=args.median, sigma_p=args.sigma_p, sigma_r=args.sigma_r, lo=64,
                  hi=args.len_hi)
    cur = make_rl_batch(shape, args.p0, args.r0, seed=args.seed, **common)
    prev = make_rl_batch(shape, args.p0, args.r0, seed=args.seed + 1, **common)
    prompt = np.repeat(np.diff(cur.prompt_offsets), args.r0)
    length = cur.max_new.reshape(-1)
    base = simulate(prompt, length, args.replicas, model)
    trainer = {"history": prev.max_new.reshape(-1), "kv_bytes_per_token": kvb, "kv_capacity": args.kv_gb * 1e9,
               "lo": 0.2, "hi": 0.5, "delta": 0.05}
    st = simulate(prompt, length, args.replicas, model, trainer=trainer)
    out = {"model": {"decode_ms": model.decode, "prefill_ms": model.prefill, "trace_records": n_rec},
           "workload": f"{args.p0} prompts x {args.r0} responses, prompt-correlated LogN(median {args.median:g}, "
                       f"sigma_p {args.sigma_p}, sigma_r {args.sigma_r}) in [64, {args.len_hi}], "
                       f"Qwen2.5-7B shape, {args.replicas} replicas",
           "rl_step_s": round(base["step_ms"] / 1e3, 3),
           "replica_end_s": [round(e / 1e3, 2) for e in base["replica_end_ms"]],
           "idle_gpu_s": round(base["idle_gpu_s"], 2), "replica_idle_frac": round(base["replica_idle_frac"], 4),
           "stream_trainer": {"rl_step_rollout_s": round(st["step_ms"] / 1e3, 3), "scaled": st["scaled"],
                              "checks": st["checks"], "train_gpu_s": round(st.get("train_gpu_s", 0.0), 2)}}
    print(json.dumps(out))


if __name__ == "__main__":
    main()
