"""FFF inference benchmark on one MI355X.

One step = one FFF forward (every step of the hot path: token load, node
logits, branch, activation, output accumulation, store) over one batch of
synthetic tokens already resident in HBM.  Default workload: one tree of
depth 11 (4095 nodes, UltraFastBERT-1x11), hidden 768, 65536 tokens, bf16
activations and weights.

Prints ONE JSON line on stdout; progress goes to stderr.  Besides the
throughput it reports:
* roofline: gathered weight bytes per launch (one W_in and one W_out row per
  visited node) over the kernel's mean launch time, against the 8 TB/s HBM
  peak, plus measured HBM traffic when a counter summary is supplied;
* dense: a dense 768 -> 3072 -> 768 GELU feedforward on the same tokens
  (bf16 hipBLASLt GEMMs with the GELU fused into the first GEMM's epilogue,
  fastest heuristic candidate), and the speedup over it;
* cpu_baseline: the fp64 CPU oracle on the host cores over a bounded sample,
  whose outputs are also compared with the device's for the same tokens.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time
from pathlib import Path

ROOT = Path(__file__).resolve().parent
if str(ROOT) not in sys.path:
    sys.path.insert(0, str(ROOT))

HBM_PEAK_GBS = 8000.0


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=None, help="a name from paper_2311_10770_amd.configs.WORKLOADS")
    ap.add_argument("--tokens", type=int, default=None, help="override the workload's token count")
    ap.add_argument("--mode", default="auto", choices=["auto", "descent", "grouped", "generic"])
    ap.add_argument("--lds-levels", type=int, default=0)
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="wall budget of the oracle timing")
    ap.add_argument("--traffic", default=None,
                    help="JSON with measured HBM bytes per launch of the FFF kernel (from rocprofv3 counters)")
    ap.add_argument("--no-check", action="store_true",
                    help="skip comparing the device output with the oracle on the CPU leg's sample")
    ap.add_argument("--copy-calib-mb", type=int, default=0,
                    help="also launch a plain copy of this many MiB 5 times (HBM counter calibration)")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the FFF layer shards by token with no exchange step, "
              "so N GPUs would each run this same one-GPU kernel on n_tokens/N tokens. "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2311_10770_amd as fff
    from paper_2311_10770_amd import benchlib, synth
    from paper_2311_10770_amd.configs import HEADLINE, WORKLOADS

    w = WORKLOADS[args.workload or HEADLINE]
    B = args.tokens or w.n_tokens
    fff.load_library()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)

    log(f"workload {w.name}: B={B} H={w.hidden} depth={w.depth} trees={w.n_trees} "
        f"x/W/y={w.x_dtype}/{w.w_dtype}/{w.y_dtype}")
    L = synth.make_layer(w.seed, B, w.hidden, w.depth, w.n_trees, w.x_dtype, w.w_dtype)
    x = fff.from_numpy(L["x"], dev)
    wi = fff.from_numpy(L["w_in"], dev)
    wo = fff.from_numpy(L["w_out"], dev)
    ydt = torch.bfloat16 if w.y_dtype == "bf16" else torch.float32
    y = torch.empty((B, w.hidden), dtype=ydt, device=dev)
    kw = dict(mode=args.mode, lds_levels=args.lds_levels)
    plan = fff.describe(x, wi, wo, w.depth, w.n_trees, y, **kw)
    log("plan:", plan)

    def step():
        fff.forward(x, wi, wo, w.depth, w.n_trees, y, **kw)

    if args.copy_calib_mb:
        src = torch.empty(args.copy_calib_mb << 20, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(5):
            benchlib.copy(src, dst)
        torch.cuda.synchronize()
        del src, dst

    t = benchlib.time_launches(step, args.steps, args.warmup, stream)
    ms = t["region_ms"] / args.steps
    tokens_per_s = B / (ms / 1e3)
    gathered = w.gathered_bytes_per_token() * B
    achieved = gathered / (t["mean_ms"] / 1e3) / 1e9
    log(f"fff: {ms * 1e3:.1f} us/step (launch mean {t['mean_ms'] * 1e3:.1f} us, std {t['std_ms'] * 1e3:.1f}), "
        f"{tokens_per_s / 1e6:.1f} M tok/s, gathered {achieved:.0f} GB/s")

    out = {
        "metric": "FFF tokens/s at d=768 depth 11; speedup vs dense 3072-FF; HBM GB/s",
        "value": tokens_per_s, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if w.w_dtype == "bf16" else "f32",
        "data": "synthetic (seeded Gaussian x ~ N(0,1), W ~ N(0,1/H); no trained weights)",
        "config": {"workload": f"FFF layer, {w.n_trees} tree(s) of depth {w.depth} "
                               f"({w.nodes} nodes), d={w.hidden}, {B} tokens, x/W/y {w.x_dtype}/{w.w_dtype}/{w.y_dtype}",
                   "name": w.name, "n_tokens": B, "hidden": w.hidden, "depth": w.depth, "n_trees": w.n_trees,
                   "mode": args.mode, "plan": plan},
        "kernel_us": {"mean": t["mean_ms"] * 1e3, "min": t["min_ms"] * 1e3, "std": t["std_ms"] * 1e3},
    }

    # Measured HBM bytes per launch from a committed counter summary, valid only while the
    # kernel sources are the ones the counters were taken on.
    from paper_2311_10770_amd.rocprof_summary import kernel_source_hash

    traffic = None
    tpath = Path(args.traffic) if args.traffic else ROOT / "profiles" / f"traffic_{w.name}_{args.mode}.json"
    if tpath.exists():
        summ = json.loads(tpath.read_text())
        if summ.get("kernel_source_hash") == kernel_source_hash():
            traffic = summ.get("hbm_bytes_per_launch")
        else:
            log(f"{tpath.name} was taken on other kernel sources: traffic unreported")
    kernels = "walk_kernel + emit_kernel" if plan.startswith("grouped") else plan.split("<")[0] + "_kernel"
    out["roofline"] = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                       "frac": achieved / HBM_PEAK_GBS, "traffic": traffic, "kernels": kernels,
                       "basis": f"gathered weight bytes per forward = {w.gathered_bytes_per_token()} B/token x {B} "
                                f"tokens, over the mean time of one forward call ({kernels}, HIP events on the "
                                f"launch stream); served by LDS/L2/MALL, not all from HBM"}
    flops = w.flops_per_token() * B
    out["alu"] = {"achieved_tflops": flops / (t["mean_ms"] / 1e3) / 1e12, "peak_tflops_fp32_vector": 157.3}

    if not args.no_dense:
        H, F = w.hidden, 3072 if w.hidden == 768 else 4 * w.hidden
        g = torch.Generator(device="cpu").manual_seed(1234)
        w1 = (torch.randn(F, H, generator=g) / H ** 0.5).to(dev, torch.bfloat16)
        w2 = (torch.randn(H, F, generator=g) / F ** 0.5).to(dev, torch.bfloat16)
        xb = x if x.dtype == torch.bfloat16 else x.to(torch.bfloat16)
        dense = benchlib.DenseFF(xb, w1, w2)
        nd = max(20, args.steps // 2)
        td = benchlib.time_launches(dense, nd, 10, stream)
        dense_ms = td["region_ms"] / nd
        # sanity: the fused-epilogue GEMMs compute the dense layer (tanh- vs erf-GELU differ slightly)
        ref = torch.nn.functional.linear(torch.nn.functional.gelu(torch.nn.functional.linear(xb[:1024].float(),
                                         w1.float())), w2.float())
        rel = float((dense.y[:1024].float() - ref).norm() / ref.norm())

        def dense_unfused():
            torch.nn.functional.linear(torch.nn.functional.gelu(torch.nn.functional.linear(xb, w1)), w2)

        tu = benchlib.time_launches(dense_unfused, nd, 5, stream)
        unfused_ms = tu["region_ms"] / nd
        out["dense"] = {"what": f"dense FF {H}->{F}->{H} on the same tokens, bf16: {dense.info}",
                        "ms": dense_ms, "tokens_per_s": B / (dense_ms / 1e3), "speedup_fff_over_dense": dense_ms / ms,
                        "rel_err_vs_fp32_torch": rel,
                        "torch_unfused_ms": unfused_ms, "speedup_fff_over_torch_unfused": unfused_ms / ms}
        dense.close()
        log(f"dense (hipBLASLt, fused GELU): {dense_ms * 1e3:.1f} us/step -> speedup {dense_ms / ms:.2f}x "
            f"(rel err {rel:.1e}); torch unfused {unfused_ms * 1e3:.1f} us")

    if not args.no_cpu_baseline:
        # The CPU leg: the fp64 oracle timed on the host cores over the first n tokens.  Its
        # outputs for those tokens are also compared with the device's (after the timed region).
        import oracle
        from oracle import parity

        threads = oracle.default_threads()
        n = min(B, 4096)
        ref = oracle.forward(L["x"][:n], L["w_in"], L["w_out"], w.depth, w.n_trees, threads=threads)
        done, t0 = 0, time.perf_counter()
        while True:
            oracle.forward(L["x"][:n], L["w_in"], L["w_out"], w.depth, w.n_trees, records=False, threads=threads)
            done += n
            if time.perf_counter() - t0 >= args.cpu_seconds:
                break
        el = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": done / el, "unit": "tokens/s", "cores": threads, "kind": "oracle",
                               "sample": f"first {n} tokens of the same batch, repeated {done // n}x over "
                                         f"{el:.1f}s wall, fp64 C oracle on {threads} host threads"}
        log(f"cpu oracle: {done / el:.0f} tok/s on {threads} threads")
        if not args.no_check:
            nodes = torch.empty((B, w.n_trees, w.depth + 1), dtype=torch.int32, device=dev)
            fff.forward(x, wi, wo, w.depth, w.n_trees, y, nodes_out=nodes, **kw)
            torch.cuda.synchronize()
            rows = np.arange(n)
            rep = parity.check(L["x"], L["w_in"], L["w_out"], w.depth, w.n_trees, ref, fff.to_numpy(y),
                               nodes.cpu().numpy(), tol=2e-2 if w.y_dtype == "bf16" else 1e-5, rows=rows)
            out["cpu_baseline"]["check"] = {"tokens": n, "ok": rep["ok"],
                                            "max_normwise_err": rep["max_normwise_err"],
                                            "n_near_tie": rep["n_near_tie"],
                                            "n_path_divergent": rep["n_path_divergent"]}
            log("device vs oracle on the sample:", out["cpu_baseline"]["check"])

    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
