"""Time every forward mode of the library over a grid of (tokens, depth[, trees]) at one hidden
size and print, per point, the mode AUTO plans and the fastest one (JSON lines).

    python -m paper_2311_10770_amd.mode_sweep --dtype bf16
    python -m paper_2311_10770_amd.mode_sweep --dtype f32 --trees 8 --depths 2,4 --tokens 1024,16384

Each mode's time is the mean of 30 calls, each between its own pair of HIP events, after 5
warm-up calls; modes that do not take the shape are reported as null.  Inputs are the seeded
synthetic layers of ``synth`` (x ~ N(0,1), W ~ N(0, 1/H)).
"""
from __future__ import annotations

import argparse
import json

import torch

from paper_2311_10770_amd import fff, synth

MODES = ("descent", "grouped", "tiled", "masked", "subtree")


def time_mode(args, kw, reps=30, warm=5) -> float:
    for _ in range(warm):
        fff.forward(*args, **kw)
    torch.cuda.synchronize()
    st = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for a, b in ev:
        a.record(st)
        fff.forward(*args, **kw)
        b.record(st)
    torch.cuda.synchronize()
    return sum(a.elapsed_time(b) for a, b in ev) / reps * 1e3


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--dtype", default="bf16", choices=["bf16", "f32"])
    ap.add_argument("--hidden", type=int, default=768)
    ap.add_argument("--trees", type=int, default=1)
    ap.add_argument("--depths", default="5,7,9,11,13")
    ap.add_argument("--tokens", default="256,1024,4096,16384,32768,65536,131072")
    args = ap.parse_args()
    dev = torch.device("cuda:0")
    toks = [int(v) for v in args.tokens.split(",")]
    for depth in (int(v) for v in args.depths.split(",")):
        L = synth.make_layer(77, max(toks), args.hidden, depth, args.trees, args.dtype, args.dtype)
        xa, wi, wo = (fff.from_numpy(L[k], dev) for k in ("x", "w_in", "w_out"))
        for B in toks:
            x = xa[:B]
            y = torch.empty_like(x)
            auto = fff.describe(x, wi, wo, depth, args.trees, y).split("<")[0]
            us = {}
            for m in MODES:
                try:
                    us[m] = round(time_mode((x, wi, wo, depth, args.trees, y), {"mode": m}), 1)
                except fff.FffError:  # the mode does not take this shape
                    us[m] = None
            best_us, best = min((v, k) for k, v in us.items() if v is not None)
            print(json.dumps({"dtype": args.dtype, "hidden": args.hidden, "trees": args.trees, "depth": depth,
                              "tokens": B, "auto": auto, "auto_us": us.get(auto), "best": best, "best_us": best_us,
                              "us": us}), flush=True)
        del xa, wi, wo, L
        torch.cuda.empty_cache()


if __name__ == "__main__":
    main()
