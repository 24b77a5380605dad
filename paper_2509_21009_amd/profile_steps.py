"""Run a few decode steps of a synthetic workload, for hardware-counter profiling.

A full rollout round launches hundreds of thousands of kernels, too many to
collect per-dispatch counters for.  This driver admits the first N
sequences of a workload, prefills them, runs a fixed number of decode steps
(all N rows live, so every projection runs with M = N), and then performs
one device-to-device copy of a known size, whose counter readings calibrate
the others.  Typical use, from the repository root:

    rocprofv3 --pmc FETCH_SIZE --kernel-include-regex "k_gemm_deep|copy" \\
        -- python3 -u paper_2509_21009_amd/profile_steps.py --workload 7b-long --seqs 64 --steps 4

All inputs are the seeded synthetic workloads of ``workloads``.
"""
from __future__ import annotations

import argparse
import os
import sys
import time

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--workload", default="7b-long")
    ap.add_argument("--seqs", type=int, default=64, help="first N sequences of the workload")
    ap.add_argument("--steps", type=int, default=4)
    ap.add_argument("--copy-mib", type=int, default=1024, help="size of the calibration copy (MiB)")
    args = ap.parse_args()

    import torch

    from paper_2509_21009_amd import rollpack as rp
    from workloads import make_weights, make_workload

    rp.load_library()
    dev = torch.device("cuda:0")
    wl = make_workload(args.workload)
    wl = wl.subset(list(range(min(args.seqs, wl.n))))
    shape = wl.shape
    weights = make_weights(shape, seed=0, device=dev)
    plens = wl.prompt_lens()
    max_new = np.maximum(wl.max_new, args.steps + 1).astype(np.int32)
    pages = int(np.sum((plens + max_new - 1 + 63) // 64)) + 16
    eng = rp.Engine(shape, rp.weights_for_engine(weights), max_seqs=wl.n,
                    max_prefill_tokens=max(16384, int(plens.max())), max_context=int(np.max(plens + max_new)),
                    kv_pages=pages)
    t0 = time.perf_counter()
    eng.prefill(wl.seq_ids, wl.prompt_tokens, wl.prompt_offsets, max_new, wl.sample_seed, wl.temperature)
    torch.cuda.synchronize()
    print(f"[profile_steps] prefilled {wl.n} sequences ({int(plens.sum())} tokens) in {time.perf_counter() - t0:.2f} s",
          flush=True)
    for i in range(args.steps):
        b, _, _ = eng.decode_step()
        torch.cuda.synchronize()
        print(f"[profile_steps] decode step {i + 1}/{args.steps}: {b} rows", flush=True)
    eng.close()
    n = args.copy_mib << 20
    src = torch.ones(n // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    print(f"[profile_steps] calibration copy of {n} bytes done", flush=True)


if __name__ == "__main__":
    main()
