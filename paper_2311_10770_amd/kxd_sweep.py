"""Speed of the UltraFastBERT-KxD family (Table 1) on one MI355X.

    python -m paper_2311_10770_amd.kxd_sweep [--dtype bf16|f32] [--tokens 16384] [--steps 20]

Every shape of Table 1 (K trees of depth D, about 4095 neurons per layer) runs
through the library's AUTO plan on the same seeded synthetic batch, so the
time can be read against the fraction of neurons a token uses, N_I/N_T =
(D+1)/(2**(D+1)-1).  The dense 768 -> 3072 -> 768 GELU feedforward (hipBLASLt
bf16, GELU fused into the first GEMM's epilogue) on the same tokens is timed
once for reference.  Prints one JSON line per shape and a summary line.
"""
from __future__ import annotations

import argparse
import json
import sys

import torch

from . import benchlib, fff, synth
from .configs import KXD_FAMILY, kxd_workload


def log(*a):
    print("[kxd]", *a, file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--dtype", default="bf16", choices=["bf16", "f32"])
    ap.add_argument("--tokens", type=int, default=16384)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--shapes", default="", help="comma list of KxD to run, e.g. 1x11,4x9 (default: all)")
    ap.add_argument("--mode", default="auto", choices=sorted(fff.MODES), help="plan to time (default: AUTO)")
    args = ap.parse_args()

    fff.load_library()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    B = args.tokens
    want = {s.strip() for s in args.shapes.split(",") if s.strip()}
    rows = []
    x = None
    for k, d in KXD_FAMILY:
        if want and f"{k}x{d}" not in want:
            continue
        w = kxd_workload(k, d, args.dtype, B)
        L = synth.make_layer(w.seed, B, w.hidden, d, k, w.x_dtype, w.w_dtype)
        x = fff.from_numpy(L["x"], dev)
        wi = fff.from_numpy(L["w_in"], dev)
        wo = fff.from_numpy(L["w_out"], dev)
        y = torch.empty((B, w.hidden), dtype=torch.bfloat16 if w.y_dtype == "bf16" else torch.float32,
                        device=dev)
        try:
            plan = fff.describe(x, wi, wo, d, k, y, mode=args.mode)
        except fff.FffError as e:
            log(f"{k}x{d}: mode {args.mode} not available ({e})")
            continue
        t = benchlib.time_launches(lambda: fff.forward(x, wi, wo, d, k, y, mode=args.mode), args.steps, args.warmup,
                                   stream)
        us = t["mean_ms"] * 1e3
        n_t, n_i = k * w.nodes, k * (d + 1)
        row = {"shape": f"{k}x{d}", "K": k, "D": d, "N_T": n_t, "N_I": n_i, "N_I_over_N_T": n_i / n_t,
               "tokens": B, "dtype": args.dtype, "us": us, "us_min": t["min_ms"] * 1e3,
               "tokens_per_s": B / (us / 1e6),
               "gathered_GBps": w.gathered_bytes_per_token() * B / (us / 1e6) / 1e9,
               "tflops": w.flops_per_token() * B / (us / 1e6) / 1e12, "plan": plan}
        rows.append(row)
        print(json.dumps(row), flush=True)
        log(f"{k}x{d}: {us:9.1f} us  {row['tokens_per_s'] / 1e6:8.1f} M tok/s  "
            f"gathered {row['gathered_GBps']:7.0f} GB/s  ({plan.split(' ')[0]})")
        del wi, wo, y

    g = torch.Generator(device="cpu").manual_seed(1234)
    H, F = 768, 3072
    w1 = (torch.randn(F, H, generator=g) / H ** 0.5).to(dev, torch.bfloat16)
    w2 = (torch.randn(H, F, generator=g) / F ** 0.5).to(dev, torch.bfloat16)
    xb = synth_x_bf16(B, H, dev)
    dense = benchlib.DenseFF(xb, w1, w2)
    td = benchlib.time_launches(dense, max(args.steps, 20), 5, stream)
    dense_us = td["mean_ms"] * 1e3
    dense.close()
    log(f"dense 768->3072->768 bf16 (hipBLASLt): {dense_us:.1f} us")
    for r in rows:
        r["speedup_over_dense"] = dense_us / r["us"]
    print(json.dumps({"summary": True, "tokens": B, "dtype": args.dtype, "dense_us": dense_us,
                      "dense": dense.info, "speedup_over_dense": {r["shape"]: r["speedup_over_dense"] for r in rows}}),
          flush=True)


def synth_x_bf16(B: int, H: int, dev):
    return fff.from_numpy(synth.make_x(6, B, H, "bf16"), dev)


if __name__ == "__main__":
    main()
