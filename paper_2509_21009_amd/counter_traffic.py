"""HBM traffic per launch of the gate/up decode GEMM from rocprofv3 counter runs.

Input: the ``--pmc FETCH_SIZE`` and ``--pmc WRITE_SIZE`` counter_collection
CSVs of ``profile_steps.py`` at 16, 32, 48 and 64 live rows (one, two, three
and four 16-row activation tiles), and the ``--kernel-trace --stats``
kernel_stats CSV of the benchmark round whose launch mix weights them.  Each
profile_steps run ends with a 1 GiB device copy; its counter readings
calibrate FETCH_SIZE and WRITE_SIZE (KiB per dispatch) to bytes.  Writes the
record bench.py reads (kernel, workload, SHA-256 of the deep kernel's source
text and launch plan, bytes per launch) and prints a table for the profile summary.  From the repository
root:

    python3 paper_2509_21009_amd/counter_traffic.py --pmc-dir results/pmc \\
        --stats results/bench_kernel_stats.csv --out profiles/gate_up_traffic.json
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re
import statistics

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SOURCE = "paper_2509_21009_amd/csrc/k_gemm.hip"
COMMON = "paper_2509_21009_amd/csrc/device_common.hpp"


def _between(text: str, start: str, end: str) -> str:
    i = text.index(start)
    return text[i:text.index(end, i) + len(end)]


def deep_source_digest(root: str = ROOT) -> str:
    """SHA-256 over what the counters measured: the k_gemm_deep kernel and its weight-load helper,
    its launch plan (the instantiated configurations and plan_deep) and the device helpers it uses.  Edits elsewhere in
    the GEMM source leave it unchanged."""
    gemm = open(os.path.join(root, SOURCE)).read()
    parts = [_between(gemm, "template <bool PACKED>\n__device__ __forceinline__ bf16x8_t load_w16", "\n}\n"),
             _between(gemm, "template <int R, int MT, int D, bool SILU, bool PACKED>\n__global__ __launch_bounds__(256) "
                            "void k_gemm_deep", "\n}\n"),
             _between(gemm, "constexpr DeepCfg kDeepCfg", "\n};\n"),
             _between(gemm, "GemmPlan plan_deep(", "\n}\n"),
             open(os.path.join(root, COMMON)).read()]
    return hashlib.sha256("\n".join(parts).encode()).hexdigest()
COPY_BYTES = 1 << 30
SHAPE = {"H": 3584, "I": 18944}  # Qwen2.5-7B hidden and intermediate sizes


def gate_up_tiles(name: str):
    """Activation tiles of a gate/up (SiLU) deep-GEMM instantiation, else None."""
    m = re.search(r"k_gemm_deep<(\d+), (\d+), (\d+), true(?:, (?:true|false))?>", name)
    return int(m.group(2)) if m else None


def read_counter(path: str, counter: str):
    rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
    copies = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]]
    gemm = {}
    for r in rows:
        t = gate_up_tiles(r["Kernel_Name"])
        if t is not None:
            gemm.setdefault(t, []).append(float(r["Counter_Value"]))
    return max(copies), gemm


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--pmc-dir", required=True)
    ap.add_argument("--stats", required=True)
    ap.add_argument("--rows", default="16,32,48,64")
    ap.add_argument("--out", default=os.path.join(ROOT, "profiles", "gate_up_traffic.json"))
    args = ap.parse_args()

    per_tile, table = {}, []
    for n in [int(x) for x in args.rows.split(",")]:
        fc, fg = read_counter(os.path.join(args.pmc_dir, f"pmc_FETCH_SIZE_{n}.csv"), "FETCH_SIZE")
        wc, wg = read_counter(os.path.join(args.pmc_dir, f"pmc_WRITE_SIZE_{n}.csv"), "WRITE_SIZE")
        fs, ws = COPY_BYTES / (fc * 1024), COPY_BYTES / (wc * 1024)
        (tiles, fvals), = fg.items()
        wvals = wg[tiles]
        fk, wk = statistics.median(fvals), statistics.median(wvals)
        read_b, write_b = fk * 1024 * fs, wk * 1024 * ws
        alg = 2 * SHAPE["I"] * SHAPE["H"] * 2 + n * SHAPE["H"] * 2 + n * SHAPE["I"] * 2
        per_tile[tiles] = read_b + write_b
        table.append((n, tiles, fk, wk, len(fvals), read_b, write_b, alg, fs, ws))
    mix = {}
    for r in csv.DictReader(open(args.stats)):
        t = gate_up_tiles(r["Name"])
        if t is not None:
            mix[t] = mix.get(t, 0) + int(r["Calls"])
    total = sum(mix.values())
    traffic = sum(per_tile[t] * c for t, c in mix.items()) / total
    alg_mix = sum((2 * SHAPE["I"] * SHAPE["H"] * 2 + 16 * t * (SHAPE["H"] + SHAPE["I"]) * 2) * c
                  for t, c in mix.items()) / total
    rec = {"kernel": "gemm_gate_up", "workload": "7b-long", "source": SOURCE,
           "source_sha256_deep": deep_source_digest(),
           "traffic_bytes_per_launch": int(round(traffic)),
           "per_tile_count": {str(t): int(round(v)) for t, v in sorted(per_tile.items())},
           "launch_mix": {str(t): c for t, c in sorted(mix.items())},
           "fetch_scale": round(table[0][8], 4), "write_scale": round(table[0][9], 4)}
    with open(args.out, "w") as f:
        json.dump(rec, f, indent=1)
    print("| live rows (M) | MFMA activation tiles | FETCH_SIZE KiB / launch (raw) | WRITE_SIZE KiB / launch (raw) "
          "| launches | HBM read, calibrated | HBM write, calibrated | algorithmic bytes | traffic / algorithmic |")
    print("|---|---|---|---|---|---|---|---|---|")
    for n, t, fk, wk, cnt, rb, wb, alg, fs, ws in table:
        print(f"| {n} | {t} | {fk:.0f} | {wk:.0f} | {cnt} | {rb / 1e6:.1f} MB | {wb / 1e6:.2f} MB | "
              f"{alg / 1e6:.1f} MB | {(rb + wb) / alg:.3f} |")
    print(f"launch mix {rec['launch_mix']}; traffic per launch {traffic / 1e6:.1f} MB against "
          f"{alg_mix / 1e6:.1f} MB algorithmic; scales fetch {table[0][8]:.4f}, write {table[0][9]:.4f}")


if __name__ == "__main__":
    main()
