"""Memory-hierarchy microbenchmarks on one MI355X: the rooflines the FFF kernels run against.

    python -m paper_2311_10770_amd.microbench

* stream read bandwidth with footprints that fit one XCD's L2, the MALL, or
  only HBM; stream write bandwidth likewise, and a copy of the output size of
  the headline layer (100.7 MB) and of 1 GiB;
* 1.5 KB row gathers by 16-lane groups (one bf16 row at hidden 768) from
  tables of those sizes, with independent row ids or a dependent chain (each
  row id computed from the previous row, like a tree walk);
* the matrix cores' issue rate for the 16x16 and 32x32 MFMA shapes in bf16 and
  fp32 at 1, 2 and 4 waves per SIMD (register operands, no memory traffic).
Prints one JSON object.
"""
from __future__ import annotations

import json
import sys

import torch

from . import benchlib


def _time(fn, reps=20, warm=3):
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(reps):
        fn()
    e.record()
    torch.cuda.synchronize()
    return s.elapsed_time(e) / reps / 1e3  # seconds


def main():
    lib = benchlib.load()
    dev = torch.device("cuda:0")
    st = torch.cuda.current_stream(dev).cuda_stream
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    big = torch.ones(2 << 30, dtype=torch.uint8, device=dev)  # 2 GiB table
    out = torch.zeros(16, dtype=torch.uint32, device=dev)
    res = {"cus": cus, "read": [], "gather": []}
    for fp in (1 << 20, 2 << 20, 16 << 20, 64 << 20, 1 << 30, 2 << 30):
        total = max(4 << 30, 4 * fp)
        for grid in (cus * 8, cus * 32):
            t = _time(lambda: lib.fffb_mb_read(big.data_ptr(), fp, total, out.data_ptr(), grid, st))
            res["read"].append({"footprint_mb": fp / 2**20, "grid": grid, "GBps": total / t / 1e9})
            print(f"read footprint {fp / 2**20:7.0f} MiB grid {grid:5d}: {total / t / 1e9:8.0f} GB/s", file=sys.stderr,
                  flush=True)
    row = 1536
    for fp in (1 << 20, 3 << 20, 12 << 20, 64 << 20, 2 << 30):
        rows = fp // row
        for dep in (0, 1):
            for groups in (cus * 16 * 4, cus * 16 * 16):
                steps = 12 if dep else 16
                t = _time(lambda: lib.fffb_mb_gather(big.data_ptr(), rows, row, groups, steps, dep, out.data_ptr(), st))
                by = groups * steps * row
                res["gather"].append({"table_mb": fp / 2**20, "dependent": dep, "groups": groups, "steps": steps,
                                      "GBps": by / t / 1e9, "us": t * 1e6})
                print(f"gather table {fp / 2**20:7.0f} MiB dep={dep} groups {groups:6d}: {by / t / 1e9:8.0f} GB/s "
                      f"({t * 1e6:.1f} us)", file=sys.stderr, flush=True)
    res["write"] = []
    for fp in (16 << 20, 128 << 20, 1 << 30, 2 << 30):
        total = max(4 << 30, 4 * fp)
        for grid in (cus * 8, cus * 32):
            if lib.fffb_mb_write(big.data_ptr(), fp, total, grid, st) != 0:
                raise RuntimeError("fffb_mb_write failed")
            t = _time(lambda: lib.fffb_mb_write(big.data_ptr(), fp, total, grid, st))
            res["write"].append({"footprint_mb": fp / 2**20, "grid": grid, "GBps": total / t / 1e9})
            print(f"write footprint {fp / 2**20:7.0f} MiB grid {grid:5d}: {total / t / 1e9:8.0f} GB/s", file=sys.stderr,
                  flush=True)
    res["copy"] = []
    for nbytes in (65536 * 768 * 2, 1 << 30):  # the headline's y (bf16) and 1 GiB
        src, dst = big[:nbytes], big[1 << 30:(1 << 30) + nbytes]
        t = _time(lambda: benchlib.copy(src, dst))
        res["copy"].append({"bytes": nbytes, "GBps_read_plus_write": 2 * nbytes / t / 1e9, "us": t * 1e6})
        print(f"copy {nbytes / 1e6:8.1f} MB: {2 * nbytes / t / 1e9:8.0f} GB/s read + write ({t * 1e6:.1f} us)",
              file=sys.stderr, flush=True)
    res["mfma"] = []
    names = {0: "16x16x32 bf16", 1: "32x32x16 bf16", 2: "16x16x4 fp32", 3: "32x32x2 fp32"}
    mout = torch.empty(cus * 4 * 256, dtype=torch.float32, device=dev)
    for shape in (0, 1, 2, 3):
        for wps in (1, 2, 4):
            flops = lib.fffb_mb_mfma(shape, cus, wps, 1000, mout.data_ptr(), st)
            if flops < 0:
                raise RuntimeError("fffb_mb_mfma failed")
            t = _time(lambda: lib.fffb_mb_mfma(shape, cus, wps, 1000, mout.data_ptr(), st))
            res["mfma"].append({"shape": names[shape], "waves_per_simd": wps, "TFLOPs": flops / t / 1e12})
            print(f"mfma {names[shape]:14s} waves/SIMD {wps}: {flops / t / 1e12:7.1f} TFLOP/s", file=sys.stderr,
                  flush=True)
    print(json.dumps(res))


if __name__ == "__main__":
    main()
