#!/usr/bin/env python3
"""Rollout benchmark on one MI355X.

A "step" is one decode step of a rollout round.  The timed region runs whole
rounds of the workload through the C ABI (rp_rollout_generate): paged-KV
admission, chunked prefill, decode steps until the longest response is done
with finished sequences freed as they go, seeded sampling and the round
metrics.  Rounds repeat until at least --steps decode steps have been timed
(one round of the default workload is 16,383 decode steps, about a minute and
a half), and `steps` in the output line counts the decode steps actually
timed.  Warm-up: every sequence of the workload is prefilled, --warmup decode
steps run at the full batch, and the sequences are aborted, all untimed.
Inputs (weights, prompts) are resident in HBM / host memory before the timed
region.

Default workload: Qwen2.5-7B shape, bf16 random weights, the long round of 64
sequences with long-tail forced response lengths (lognormal, median 4096,
sigma 1.0, clamped to [512, 16384]), temperature 1.0.

Prints one JSON line.  `--gpus N` with N > 1 is refused: the benchmark
measures one GPU (data-parallel replicas are independent engines, one process
per GPU, each with its own share of the sequences).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode tokens/s/GPU + % peak HBM BW, Qwen2.5-7B-shape long-tail rollout"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFS = 2500.0  # dense bf16 MFMA, MI355X
PREFILL_GEMMS = ["gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down"]
BF16_PEAK_TFLOPS = 2500.0
WORKLOAD_TEXT = {
    "7b-long": "Qwen2.5-7B shape long round: 64 seqs, prompts U[128,1024], responses LogN(4096, 1.0) "
               "clamped [512,16384], forced lengths, T=1.0",
    "7b-short": "Qwen2.5-7B shape short round: 512 seqs, prompts U[128,1024], responses LogN(768, 0.4) "
                "clamped [64,2048], T=1.0",
    "7b-mixed": "Qwen2.5-7B shape: short round (512 seqs) then long round (64 seqs), given round ids",
    "0.5b": "Qwen2.5-0.5B shape: 32 prompts x 8 responses, prompts U[64,512], LogN(512, 0.8) clamped "
            "[32,4096], T=1.0",
    "32b": "Qwen2.5-32B shape: 96 seqs, prompts U[256,1024], LogN(2048, 0.9) clamped [64,8192], T=1.0",
    "tiny": "tiny fp32 decoder: 8 prompts x 32 tokens, 64 greedy tokens each",
}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def decode_bytes_model(shape, prompt_lens, max_new):
    """Algorithmic HBM bytes of every decode step of one round: the weights
    once per step plus the K/V of every attended token."""
    wbytes = shape.decode_weight_bytes()
    kvb = shape.kv_bytes_per_token()
    p = np.asarray(prompt_lens, np.int64)
    L = np.asarray(max_new, np.int64)
    steps = int(L.max()) - 1
    total = 0.0
    for j in range(1, steps + 1):
        act = L > j
        total += wbytes + float(np.sum(p[act] + j)) * kvb
    return total, steps


EMBED_ROWS = 1024


def live_rows_per_step(wl):
    """Rows (live sequences) of every decode step of the workload's rounds, in order."""
    rounds = [np.arange(wl.n)] if wl.round_id is None else [np.flatnonzero(wl.round_id == r)
                                                             for r in sorted(set(wl.round_id.tolist()))]
    rows = []
    for idx in rounds:
        L = np.sort(np.asarray(wl.max_new[idx], np.int64))
        j = np.arange(1, int(L[-1]))
        rows.append(len(L) - np.searchsorted(L, j, side="right"))
    return np.concatenate(rows)


def cpu_baseline(weights, shape, wl):
    """Time the oracle on a bounded sample and scale it to generated tokens/s.

    Sample: full-batch decode steps of the oracle (oracle.model.decode_step_batch:
    one step for B sequences, [B, H] products) through the first layer plus the
    LM head, at B = every sequence of the workload, 64, 8 and 1; the caches hold
    the rows' real prompt lengths of random keys and values (the step's work
    depends on their lengths only).  One prefill of the shortest prompt through
    the first layer (KVState.step, which also computes the LM head of every
    prompt position) is timed too.  The per-layer share is scaled to all layers,
    and the round is extrapolated step by step with each step's live row count
    (times interpolated linearly in B between the measured batches).
    """
    from threadpoolctl import threadpool_info

    from oracle import model as om
    from workloads import truncated, weights_to_numpy

    t_sample0 = time.perf_counter()
    # An untied model reads the embedding only at the sample's token ids: the sample converts its first
    # EMBED_ROWS rows and takes token ids below that (the work does not depend on the ids).
    n_emb = shape.vocab if weights["lm_head"] is None else min(EMBED_ROWS, shape.vocab)
    sub = {"embed": weights["embed"][:n_emb], "final_norm": weights["final_norm"], "lm_head": weights["lm_head"],
           "layers": weights["layers"][:1]}
    w64 = weights_to_numpy(sub)
    t_convert = time.perf_counter() - t_sample0
    s1 = truncated(shape, 1)
    plens = wl.prompt_lens()
    rng = np.random.default_rng(0)

    def states_for(idx):
        sts = []
        for i in idx:
            st = om.KVState(s1)
            n = int(plens[i])
            st.k[0] = rng.standard_normal((n, shape.n_kv, shape.head_dim)) * 0.5
            st.v[0] = rng.standard_normal((n, shape.n_kv, shape.head_dim)) * 0.5
            st.length = n
            sts.append(st)
        return sts

    def best_of(reps, fn):
        ts = []
        for _ in range(reps):
            t0 = time.perf_counter()
            fn()
            ts.append(time.perf_counter() - t0)
        return min(ts)

    batches = sorted({b for b in (wl.n, 64, 8, 1) if b <= wl.n})
    om.decode_step_batch(w64, states_for([0]), [0])  # first call: thread pools and first touch, untimed
    t_full, t_lm = {}, {}
    for B in batches:
        idx = np.arange(B)
        sts = states_for(idx)
        toks = np.array([wl.prompt(i)[-1] for i in idx]) % n_emb
        t_step1 = best_of(2, lambda: om.decode_step_batch(w64, sts, toks))
        x = rng.standard_normal((B, shape.hidden))
        t_lm[B] = best_of(2, lambda: om.lm_head(w64, x, s1))
        t_full[B] = shape.layers * max(t_step1 - t_lm[B], 0.0) + t_lm[B]
    bs = np.array(batches, np.float64)
    tf = np.array([t_full[b] for b in batches])
    decode_t = float(np.sum(np.interp(live_rows_per_step(wl), bs, tf)))
    # prefill of the shortest prompt through layer 0 (with the oracle's LM head over every position)
    i0 = int(np.argmin(plens))
    st = om.KVState(s1)
    t0 = time.perf_counter()
    st.step(w64, wl.prompt(i0) % n_emb)
    t_pre = time.perf_counter() - t0
    p0 = int(plens[i0])
    t0 = time.perf_counter()
    om.lm_head(w64, rng.standard_normal((p0, shape.hidden)), s1)
    t_pre_lm = time.perf_counter() - t0
    per_tok = (shape.layers * max(t_pre - t_pre_lm, 0.0) + t_pre_lm) / p0
    prefill_t = float(np.sum(plens)) * per_tok
    total_t = decode_t + prefill_t
    gen = int(np.sum(wl.max_new))
    threads = sum(int(i.get("num_threads", 0)) for i in threadpool_info() if i.get("user_api") == "blas") or 1
    return {"value": round(gen / total_t, 3), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": (f"fp64 numpy oracle (oracle.model.decode_step_batch), full-batch decode steps through layer 0 "
                       f"+ LM head at B = {batches} (s/step scaled to {shape.layers} layers: "
                       + ", ".join(f"B={b}: {t_full[b]:.2f}" for b in batches)
                       + f"), plus a {p0}-token prefill through layer 0; extrapolated over the "
                       f"{len(live_rows_per_step(wl))} decode steps of the workload ({gen} tokens) with each step's "
                       f"live rows: decode {decode_t:.0f} s + prefill {prefill_t:.0f} s; host cpus "
                       f"{len(os.sched_getaffinity(0))}; sample took {time.perf_counter() - t_sample0:.1f} s, of which "
                       f"{t_convert:.1f} s converting the sampled weights to fp64"),
            "extrapolated": True}


TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "gate_up_traffic.json")


def measured_traffic(kernel: str, workload: str, path: str = TRAFFIC_RECORD):
    """HBM bytes per launch of the roofline kernel from the calibrated FETCH_SIZE / WRITE_SIZE
    counter runs recorded in profiles/, or None when there is no record for this kernel and
    workload or the kernel (its source text and launch plan) has changed since the counters were
    taken."""
    from paper_2509_21009_amd.counter_traffic import deep_source_digest
    try:
        with open(path) as f:
            rec = json.load(f)
        digest = deep_source_digest(ROOT)
    except (OSError, ValueError, KeyError):
        return None
    if rec.get("kernel") != kernel or rec.get("workload") != workload or rec.get("source_sha256_deep") != digest:
        return None
    return int(rec["traffic_bytes_per_launch"])


def measured_stream_gbs(gib: float = 2.0, reps: int = 5) -> float:
    """The practical HBM read ceiling on this device (rp_stream_read_gbs: the library's streaming
    read kernel over a `gib` GiB buffer, far past the 256 MB last-level cache, fastest of `reps`)."""
    import torch
    from paper_2509_21009_amd import rollpack as rp
    x = torch.empty(int(gib * (1 << 30)), dtype=torch.uint8, device="cuda")
    x.fill_(1)
    gbs = rp.rp_stream_read_gbs(x, reps)
    del x
    torch.cuda.empty_cache()
    return gbs


DECODE_GEMMS = PREFILL_GEMMS + ["gemm_lm_head"]
FULL_BATCH_DECODE_STEPS = 8


def gemm_rates(eng, wl):
    """MFMA utilisation of the prefill projections and of the decode GEMMs at the round's full batch,
    from HIP events on the engine's stream: one untimed prefill of every prompt of the workload (in
    chunks of max_prefill_tokens), then FULL_BATCH_DECODE_STEPS decode steps with every sequence
    live, the sequences then aborted.  flops are 2*M*N*K per launch, bytes the algorithmic
    weights + activations + outputs."""
    import torch
    eng.profile(PREFILL_GEMMS + ["attn"])
    eng.prefill(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, np.maximum(wl.max_new, 2).astype(np.int32),
                wl.sample_seed, wl.temperature)
    torch.cuda.synchronize()
    allp = eng.profile_read()
    prof = [p for p in allp if p["phase"] == "prefill" and p["kernel"] in PREFILL_GEMMS]
    attn = [p for p in allp if p["phase"] == "prefill" and p["kernel"] == "attn"]
    eng.profile(DECODE_GEMMS)
    # steps before the first sequence could finish, so the batch stays whole
    steps = max(1, min(FULL_BATCH_DECODE_STEPS, int(np.maximum(wl.max_new, 2).min()) - 1))
    for _ in range(steps):
        eng.decode_step()
    torch.cuda.synchronize()
    dec = [p for p in eng.profile_read() if p["phase"] == "decode" and p["kernel"] in DECODE_GEMMS]
    eng.profile([])
    eng.abort(wl.seq_ids)
    eng.free_finished()

    def rates(ps):
        flops = sum(p["flops"] for p in ps)
        ms = sum(p["total_ms"] for p in ps)
        if ms <= 0:
            return None
        tfs = flops / (ms * 1e-3) / 1e12
        return {"achieved": round(tfs, 1), "peak": MFMA_BF16_PEAK_TFS, "unit": "TFLOP/s",
                "frac": round(tfs / MFMA_BF16_PEAK_TFS, 4),
                "hbm_gbs": round(sum(p["bytes"] for p in ps) / (ms * 1e-3) / 1e9, 1),
                "per_kernel_tflops": {p["kernel"]: round(p["flops"] / (p["total_ms"] * 1e-3) / 1e12, 1) for p in ps}}

    pre = rates(prof)
    if pre is not None:
        pre["prompt_tokens"] = int(wl.prompt_lens().sum())
    full = rates(dec)
    if full is not None:
        full["rows"] = int(wl.n)
        full["steps"] = steps
    att = rates(attn)
    if att is not None:
        att.pop("per_kernel_tflops", None)
        att["flops"] = "2 n_q hd sum_i p_i(p_i + 1): the causal products only"
    return pre, full, att


def warmup_steps(eng, wl, n_steps):
    """Untimed: prefill every sequence of the workload, run n_steps decode steps at the full
    batch, then abort the sequences."""
    if n_steps <= 0:
        return
    eng.prefill(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, np.maximum(wl.max_new, 2).astype(np.int32),
                wl.sample_seed, wl.temperature)
    for _ in range(n_steps):
        eng.decode_step()
    eng.abort(wl.seq_ids)
    eng.free_finished()


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1,
                    help="decode steps to time, at least: whole rounds run until this many have been timed")
    ap.add_argument("--warmup", type=int, default=4, help="untimed decode steps at the full batch first")
    ap.add_argument("--workload", default="7b-long", choices=sorted(WORKLOAD_TEXT))
    ap.add_argument("--kernel", default="gemm_gate_up", help="kernel class whose roofline is reported")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gemm-rates", action="store_true",
                    help="skip the MFMA-utilisation pass (prefill projections, decode GEMMs at the full batch)")
    ap.add_argument("--profile-every", type=int, default=8,
                    help="time one launch in N of the roofline kernel inside the timed rounds (1: all)")
    ap.add_argument("--class-rates", action="store_true",
                    help="time every kernel class (one launch in --profile-every) inside the timed rounds and report "
                         "each class's decode rate in config.decode_class_rates (slows the rounds by a few percent)")
    ap.add_argument("--max-prefill-tokens", type=int, default=16384)
    ap.add_argument("--step-trace", default=None, metavar="PATH",
                    help="after the timed steps, run one more (untimed) round with the per-step trace on and write "
                         "its records (kind, round, rows, summed context, ms) to PATH as JSON")
    ap.add_argument("--compare-unscheduled", action="store_true",
                    help="after the timed steps, run the same sequences as one unscheduled batch and report "
                         "both schedules (meaningful for 7b-mixed: short round + long round vs one batch)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on exactly one GPU (got --gpus {args.gpus}, WORLD_SIZE {world}); "
              "data-parallel replicas are independent engines, one process per GPU, and are not run here.",
              file=sys.stderr)
        sys.exit(2)
    t_start = time.perf_counter()

    import torch

    from paper_2509_21009_amd import rollpack as rp
    from workloads import make_weights, make_workload

    if not os.path.exists(rp.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    rp.load_library()
    dev = torch.device("cuda:0")
    wl = make_workload(args.workload)
    shape = wl.shape
    log(f"workload {args.workload}: {wl.n} seqs, {int(wl.max_new.sum())} new tokens, max {int(wl.max_new.max())}")
    t0 = time.perf_counter()
    weights = make_weights(shape, seed=0, device=dev)
    torch.cuda.synchronize()
    log(f"weights generated in {time.perf_counter() - t0:.1f} s")
    wd = rp.weights_for_engine(weights)
    plens = wl.prompt_lens()
    need_ctx = int(np.max(plens + wl.max_new))
    pages = int(np.sum((plens + wl.max_new - 1 + 63) // 64)) + 16
    eng = rp.Engine(shape, wd, max_seqs=wl.n, max_prefill_tokens=max(args.max_prefill_tokens, int(plens.max())),
                    max_context=need_ctx, kv_pages=pages)
    call = lambda: eng.rollout(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, wl.max_new, wl.sample_seed,  # noqa
                               wl.temperature, wl.round_id)
    t0 = time.perf_counter()
    warmup_steps(eng, wl, args.warmup)
    torch.cuda.synchronize()
    log(f"warm-up: prefill + {args.warmup} decode steps at {wl.n} rows in {time.perf_counter() - t0:.1f} s")
    eng.profile(list(rp.KERNEL_CLASSES) if args.class_rates else [args.kernel], every=args.profile_every)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    all_stats = []
    timed_steps = 0
    while timed_steps < max(args.steps, 1):
        _, stats = call()
        all_stats.append(stats)
        timed_steps += sum(int(s["decode_steps"]) for s in stats)
        log(f"timed round set {len(all_stats)}: " + ", ".join(
            f"round {s['round_id']}: {s['makespan_ms'] / 1e3:.2f} s, {s['decode_steps']} decode steps" for s in stats))
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    prof = eng.profile_read()
    eng.profile([])

    n_sets = len(all_stats)
    gen_tokens = int(wl.max_new.sum()) * n_sets
    value = gen_tokens / elapsed
    last = all_stats[-1]
    decode_s = sum(s["decode_ms"] for s in last) / 1e3
    makespan_s = sum(s["makespan_ms"] for s in last) / 1e3
    dec_bytes = 0.0
    rounds = [np.arange(wl.n)] if wl.round_id is None else [np.flatnonzero(wl.round_id == r)
                                                             for r in sorted(set(wl.round_id.tolist()))]
    for idx in rounds:
        b, _ = decode_bytes_model(shape, plens[idx], wl.max_new[idx])
        dec_bytes += b
    dec = [p for p in prof if p["phase"] == "decode" and p["kernel"] == args.kernel]
    roof = None
    if dec:
        p = dec[0]
        avg_ms = p["total_ms"] / p["launches"]
        bytes_per = p["bytes"] / p["launches"]
        achieved = bytes_per / (avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(args.kernel, args.workload),
                "kernel": args.kernel,
                "phase": "decode", "launches": p["launches"], "timed_every": args.profile_every,
                "avg_launch_us": round(avg_ms * 1e3, 2),
                "algorithmic_bytes_per_launch": bytes_per}
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": timed_steps,
        "warmup": args.warmup, "ms_per_step": round(elapsed * 1e3 / timed_steps, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": shape.dtype, "data": "synthetic",
        "config": {"workload": WORKLOAD_TEXT[args.workload], "sequences": wl.n,
                   "step": "one decode step; the timed region is whole rounds (prefill, decode, sampling, freeing)",
                   "requested_steps": args.steps, "timed_round_sets": n_sets, "timed_s": round(elapsed, 3),
                   "generated_tokens_per_round_set": int(wl.max_new.sum()),
                   "prompt_tokens_per_round_set": int(plens.sum()),
                   "makespan_s": round(makespan_s, 3), "decode_s": round(decode_s, 3),
                   "decode_tokens_per_s": round(int(wl.max_new.sum()) / max(decode_s, 1e-9), 1),
                   "decode_hbm_frac": round(dec_bytes / max(decode_s, 1e-9) / (HBM_PEAK_GBS * 1e9), 4),
                   "rounds": [{k: (round(v, 4) if isinstance(v, float) else v) for k, v in s.items()} for s in last]},
        "roofline": roof,
    }
    if args.class_rates:
        out["config"]["decode_class_rates"] = {
            p["kernel"]: {"timed_launches": p["launches"], "avg_us": round(p["total_ms"] * 1e3 / p["launches"], 2),
                          "gbs": round(p["bytes"] / (p["total_ms"] * 1e-3) / 1e9, 1),
                          "tflops": round(p["flops"] / (p["total_ms"] * 1e-3) / 1e12, 1)}
            for p in prof if p["phase"] == "decode" and p["launches"] > 0}
    if n_sets > 1:
        out["config"]["round_makespan_median_s"] = round(float(np.median(
            [sum(s_["makespan_ms"] for s_ in st) / 1e3 for st in all_stats])), 3)
    log(f"timed: {timed_steps} decode steps in {elapsed:.2f} s, {value:.1f} tokens/s")
    if roof is not None:
        stream = measured_stream_gbs()
        roof["measured_peak"] = round(stream, 1)
        roof["frac_measured"] = round(roof["achieved"] / stream, 4)
    if shape.dtype == "bf16" and not args.no_gemm_rates:
        t0 = time.perf_counter()
        (out["config"]["prefill_gemm_mfma"], out["config"]["decode_gemm_full_batch"],
         out["config"]["prefill_attn_mfma"]) = gemm_rates(eng, wl)
        log(f"GEMM rate pass in {time.perf_counter() - t0:.1f} s")
    if args.compare_unscheduled and wl.round_id is not None:
        log("running the same sequences as one unscheduled batch")
        _, flat = eng.rollout(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, wl.max_new, wl.sample_seed,
                              wl.temperature, None)
        sched_make = sum(s_["makespan_ms"] for s_ in last) / 1e3
        sched_idle = sum(s_["idle_slot_s"] for s_ in last)
        out["config"]["schedule_comparison"] = {
            "rounds_makespan_s": round(sched_make, 3), "rounds_idle_slot_s": round(sched_idle, 1),
            "unscheduled_makespan_s": round(flat[0]["makespan_ms"] / 1e3, 3),
            "unscheduled_idle_slot_s": round(flat[0]["idle_slot_s"], 1),
            "unscheduled_slot_idle": round(flat[0]["slot_idle"], 4),
            "idle_reduction": round(flat[0]["idle_slot_s"] / max(sched_idle, 1e-9), 3)}
    if args.step_trace:
        log("running one more round with the per-step trace")
        eng.step_trace(1 << 20)
        call()
        rec = eng.step_trace_read()
        eng.step_trace(0)
        with open(args.step_trace, "w") as f:
            json.dump({"workload": args.workload, "model": shape.name, "fields": ["kind", "round_id", "rows",
                                                                                 "sum_ctx", "ms"],
                       "records": [[int(r["kind"]), int(r["round_id"]), int(r["rows"]), int(r["sum_ctx"]),
                                    round(float(r["ms"]), 5)] for r in rec]}, f)
        log(f"step trace: {len(rec)} records written to {args.step_trace}")
    eng.close()
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a sample")
        t0 = time.perf_counter()
        out["cpu_baseline"] = cpu_baseline(weights, shape, wl)
        log(f"CPU oracle sample in {time.perf_counter() - t0:.1f} s")
    out["config"]["process_s"] = round(time.perf_counter() - t_start, 1)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
