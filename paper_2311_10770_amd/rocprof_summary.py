"""Summarise rocprofv3 CSV output for the kernels of one FFF step: mean
duration from a kernel-trace stats file, and HBM bytes per dispatch from
FETCH_SIZE / WRITE_SIZE counter runs, scaled by what the same counters read
for the plain copy kernel of known size launched beside it (bench.py
--copy-calib-mb).  ``--kernel`` takes comma-separated name fragments; a step
launches each named kernel once, so per-step figures are their sums.

    python -m paper_2311_10770_amd.rocprof_summary --kernel walk_kernel,emit_kernel \\
        --stats DIR/kernel_stats.csv --fetch DIR_F/counter_collection.csv \\
        --write DIR_W/counter_collection.csv --copy-mb 512 --out summary.json
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
from pathlib import Path

PKG = Path(__file__).resolve().parent
COPY_KERNEL = "copy_kernel"


def kernel_source_hash(backward: bool = False) -> str:
    """Hash of the sources the forward (or backward) kernels are compiled from: counter figures
    taken on them are void once these change."""
    h = hashlib.sha256()
    main = "fff_backward.hip" if backward else "fff_kernels.hip"
    for name in (main, "fff_common.hpp", "fff_device.hpp", "fff_internal.hpp"):
        p = PKG / "csrc" / name
        if p.exists():
            h.update(p.read_bytes())
    return h.hexdigest()[:16]


def read_stats(path: Path, kernel: str) -> dict:
    rows = list(csv.DictReader(open(path)))
    for r in rows:
        if kernel in r["Name"]:
            return {"name": r["Name"], "calls": int(r["Calls"]), "mean_us": float(r["AverageNs"]) / 1e3,
                    "min_us": float(r["MinNs"]) / 1e3, "max_us": float(r["MaxNs"]) / 1e3}
    raise KeyError(f"{kernel} not in {path}")


def read_counter(path: Path, counter: str, kernel: str) -> list:
    vals = []
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] == counter and kernel in r["Kernel_Name"]:
            vals.append(float(r["Counter_Value"]))
    if not vals:
        raise KeyError(f"no {counter} rows for {kernel} in {path}")
    return vals


HBM_PEAK_GBS = 8000.0


def summarise(kernels: str, stats: Path | None, fetch: Path | None, write: Path | None, copy_mb: int,
              algorithmic: str | None = None) -> dict:
    names = [k for k in kernels.split(",") if k]
    out = {"kernels": names, "kernel_source_hash": kernel_source_hash(any(k.startswith("bwd_") for k in names))}
    if stats:
        durs = [read_stats(stats, k) for k in names]
        out["duration"] = {"per_kernel": durs, "step_mean_us": sum(d["mean_us"] for d in durs)}
    copy_bytes = copy_mb * (1 << 20)
    total = 0.0
    for what, path in (("FETCH_SIZE", fetch), ("WRITE_SIZE", write)):
        if not path:
            continue
        c = read_counter(path, what, COPY_KERNEL)
        c_kib = sum(c) / len(c)
        scale = copy_bytes / (c_kib * 1024.0)  # true bytes per counted byte, from the copy
        per = {}
        for k in names:
            v = read_counter(path, what, k)
            per[k] = {"kib_per_dispatch": sum(v) / len(v), "dispatches": len(v),
                      "bytes_per_dispatch": sum(v) / len(v) * 1024.0 * scale}
        step = sum(d["bytes_per_dispatch"] for d in per.values())
        out[what] = {"copy_kib_per_dispatch": c_kib, "copy_true_bytes": copy_bytes, "scale": scale,
                     "per_kernel": per, "bytes_per_step": step}
        total += step
    if fetch and write:
        out["hbm_bytes_per_launch"] = total
    if algorithmic:
        # per kernel: the bytes it cannot avoid (given), the bytes the counters saw, their ratio, and
        # the algorithmic bytes over its mean duration against the 8 TB/s HBM peak
        algo = [float(v) for v in algorithmic.split(",")]
        if len(algo) != len(names):
            raise ValueError("--algorithmic needs one byte count per --kernel name")
        table = []
        for i, k in enumerate(names):
            row = {"kernel": k, "algorithmic_bytes": algo[i]}
            if "FETCH_SIZE" in out and "WRITE_SIZE" in out:
                cb = out["FETCH_SIZE"]["per_kernel"][k]["bytes_per_dispatch"] + \
                    out["WRITE_SIZE"]["per_kernel"][k]["bytes_per_dispatch"]
                row["counter_bytes"] = cb
                row["counter_over_algorithmic"] = cb / algo[i] if algo[i] else None
            if stats:
                us = out["duration"]["per_kernel"][i]["mean_us"]
                row["mean_us"] = us
                row["algorithmic_gbs"] = algo[i] / (us * 1e-6) / 1e9
                row["frac_of_hbm_peak"] = row["algorithmic_gbs"] / HBM_PEAK_GBS
            table.append(row)
        out["per_kernel_roofline"] = table
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--kernel", required=True)
    ap.add_argument("--stats", type=Path)
    ap.add_argument("--fetch", type=Path)
    ap.add_argument("--write", type=Path)
    ap.add_argument("--copy-mb", type=int, default=512)
    ap.add_argument("--out", type=Path)
    ap.add_argument("--algorithmic", default=None,
                    help="comma-separated algorithmic bytes per dispatch, one per --kernel name")
    a = ap.parse_args()
    s = summarise(a.kernel, a.stats, a.fetch, a.write, a.copy_mb, a.algorithmic)
    text = json.dumps(s, indent=1)
    if a.out:
        a.out.write_text(text + "\n")
    print(text)


if __name__ == "__main__":
    main()
