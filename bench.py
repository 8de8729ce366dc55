"""FFF inference benchmark on one MI355X.

One step = one FFF forward (every step of the hot path: token load, node
logits, branch, activation, output accumulation, store) over one batch of
synthetic tokens already resident in HBM.  Default workload: one tree of
depth 11 (4095 nodes, UltraFastBERT-1x11), hidden 768, 65536 tokens, bf16
activations and weights.

Prints ONE JSON line on stdout; progress goes to stderr.  Besides the
throughput it reports:
* roofline: the compulsory HBM bytes of one forward (x read once, y written
  once, every weight row the batch touches read once) over the mean forward
  time of the timed region, against the 8 TB/s HBM peak, with the HBM bytes
  the counters measured (a committed rocprofv3 summary) beside them;
* gathered: the weight bytes the walk and the emit read per token (one W_in
  and one W_out row per visited node) over the same time -- served mostly by
  LDS, L2 and MALL, so this rate exceeds the HBM peak;
* valu_only: the same layer through the vector-ALU plan (grouped or fused
  descent, no matrix cores) when the default plan uses MFMA;
* dense: a dense 768 -> 3072 -> 768 GELU feedforward on the same tokens
  (hipBLASLt GEMMs with the GELU fused into the first GEMM's epilogue,
  fastest heuristic candidate; bf16, and fp32 for fp32 workloads), its
  achieved rate against the MFMA peak, and the speedups over it;
* paper: the paper's own speedups, with the hardware they were measured on;
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
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}  # dense MI355X peaks (no sparsity)

# The paper's speedups of the FFF over a dense feedforward (Section 3.3, Table 2), with the
# hardware and software they were measured on; context for the MI355X figures, not targets.
PAPER_SPEEDUPS = {
    "fff_cpu_level2_over_fastest_dense_cpu": {
        "value": 78.0, "hardware": "Intel Core i7-6700HQ, Intel MKL 2023.2.0, 64-bit routines",
        "what": "FFF through batched BLAS level-2 routines vs the fastest dense feedforward (level-3 GEMM)"},
    "fff_pytorch_bmm_over_dense_same_primitive": {
        "value": 39.45, "hardware": "NVIDIA RTX A6000, CUDA 11.7, PyTorch 2.0.1",
        "what": "FFF through PyTorch batched matmul vs FF-4095 through the same primitive (the abstract's 40x)"},
    "fff_pytorch_bmm_over_fastest_dense_gpu": {
        "value": 3.15, "hardware": "NVIDIA RTX A6000, CUDA 11.7, PyTorch 2.0.1",
        "what": "FFF through PyTorch batched matmul vs the fastest dense feedforward (native fused)"},
    "theoretical_limit": {"value": 341.25, "hardware": "analytic", "what": "4095 neurons / 12 used per token"},
}


def host_cpu() -> str:
    """Host CPU model and logical CPU count, from /proc/cpuinfo."""
    model, count = "unknown", 0
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                count += 1
    except OSError:
        pass
    return f"{model} ({count} logical CPUs)"


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=None, help="a name from paper_2311_10770_amd.configs.WORKLOADS")
    ap.add_argument("--tokens", type=int, default=None, help="override the workload's token count")
    ap.add_argument("--mode", default="auto", choices=["auto", "descent", "grouped", "tiled", "generic", "masked", "subtree"])
    ap.add_argument("--lds-levels", type=int, default=0)
    ap.add_argument("--norm", action="store_true", help="LayerNorm before every layer (gain/shift drawn per layer)")
    ap.add_argument("--backward", action="store_true",
                    help="time the hard-routed backward (dx, dW_in, dW_out from the forward's records) instead")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-valu-only", action="store_true",
                    help="skip timing the vector-ALU plan beside an MFMA plan (keeps a profile to one plan)")
    ap.add_argument("--cold-reps", type=int, default=20,
                    help="calls timed cold (a 1 GiB write before each evicts W from L2 and MALL); 0: skip")
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

    NL = w.layers
    log(f"workload {w.name}: B={B} H={w.hidden} depth={w.depth} trees={w.n_trees} layers={NL} "
        f"x/W/y={w.x_dtype}/{w.w_dtype}/{w.y_dtype} norm={args.norm}")
    kw = dict(mode=args.mode, lds_levels=args.lds_levels)
    if NL == 1:
        L = synth.make_layer(w.seed, B, w.hidden, w.depth, w.n_trees, w.x_dtype, w.w_dtype)
        layers_np = [{"w_in": L["w_in"], "w_out": L["w_out"]}]
    else:
        # a stack: layer i's weights (and LayerNorm parameters) are drawn with layer index i + 1
        L = {"x": synth.make_x(w.seed, B, w.hidden, w.x_dtype)}
        layers_np = []
        for i in range(NL):
            wi_np, wo_np = synth.make_weights(w.seed, w.hidden, w.depth, w.n_trees, w.w_dtype, layer=i + 1)
            layers_np.append({"w_in": wi_np, "w_out": wo_np})
    if args.norm:
        for i, lay in enumerate(layers_np):
            lay["gamma"], lay["beta"] = synth.make_norm(w.seed, w.hidden, layer=i + 1 if NL > 1 else 0)
        kw.update(norm="layernorm", norm_eps=1e-12)
    x = fff.from_numpy(L["x"], dev)
    dlayers = [tuple(fff.from_numpy(lay[k], dev) for k in ("w_in", "w_out", "gamma", "beta") if k in lay)
               for lay in layers_np]
    wi, wo = dlayers[0][0], dlayers[0][1]
    ydt = torch.bfloat16 if w.y_dtype == "bf16" else torch.float32
    y = torch.empty((B, w.hidden), dtype=ydt, device=dev)

    def layer_kw(i):
        if not args.norm:
            return {}
        return dict(norm_gamma=dlayers[i][2], norm_beta=dlayers[i][3])

    if args.backward:
        if NL != 1 or args.norm:
            sys.exit("--backward times one layer without LayerNorm")
        rec = (B, w.n_trees, w.depth + 1)
        nodes_rec = torch.empty(rec, dtype=torch.int32, device=dev)
        logits_rec = torch.empty(rec, dtype=torch.float32, device=dev)
        fff.forward(x, wi, wo, w.depth, w.n_trees, y, nodes_out=nodes_rec, logits_out=logits_rec, **kw)
        leaves = nodes_rec[:, :, w.depth].contiguous()
        dy = fff.from_numpy(synth.make_x(w.seed + 100, B, w.hidden, w.y_dtype), dev)
        dx = torch.empty_like(x)
        nn_ = (1 << (w.depth + 1)) - 1
        dwi = torch.empty((w.n_trees, nn_, w.hidden), dtype=torch.float32, device=dev)
        dwo = torch.empty_like(dwi)
        fused = (w.n_trees == 1 and w.w_dtype == "bf16" and w.depth <= 15 and w.hidden % 128 == 0
                 and w.hidden <= 1024)
        plan = ("backward: stable sort by leaf (rank, leaf sums, base, place) + fused leaf-tiled kernel "
                "(da, dx, dW on MFMA per 16-token tile) + sums of the rows above the subtrees" if fused else
                "backward: token kernel + stable sort by leaf + weight kernel + fix-up sums")

        def step():
            fff.backward(x, wi, wo, w.depth, w.n_trees, dy, leaves, logits_rec, dx=dx, dw_in=dwi, dw_out=dwo,
                         act="gelu")
    elif NL == 1:
        plan = fff.describe(x, wi, wo, w.depth, w.n_trees, y, **kw, **layer_kw(0))

        def step():
            fff.forward(x, wi, wo, w.depth, w.n_trees, y, **kw, **layer_kw(0))
    else:
        plan = fff.describe_stack(x, dlayers, w.depth, w.n_trees, y, **kw)

        def step():
            fff.forward_stack(x, dlayers, w.depth, w.n_trees, y, **kw)
    log("plan:", plan)

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
    gathered = w.gathered_bytes_per_token() * B * NL
    achieved = gathered / (t["mean_ms"] / 1e3) / 1e9
    log(f"fff: {ms * 1e3:.1f} us/step (launch mean {t['mean_ms'] * 1e3:.1f} us, std {t['std_ms'] * 1e3:.1f}), "
        f"{tokens_per_s / 1e6:.1f} M tok/s, gathered {achieved:.0f} GB/s")

    out = {
        "metric": ("FFF hard-routed backward tokens/s (dx, dW_in, dW_out)" if args.backward else
                   "FFF tokens/s at d=768 depth 11; speedup vs dense 3072-FF; HBM GB/s"),
        "value": tokens_per_s, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if w.w_dtype == "bf16" else "f32",
        "data": "synthetic (seeded Gaussian x ~ N(0,1), W ~ N(0,1/H); no trained weights)",
        "config": {"workload": (f"{NL} stacked " if NL > 1 else "") +
                               f"FFF layer{'s' if NL > 1 else ''}{' with LayerNorm' if args.norm else ''}, "
                               f"{w.n_trees} tree(s) of depth {w.depth} "
                               f"({w.nodes} nodes), d={w.hidden}, {B} tokens, x/W/y {w.x_dtype}/{w.w_dtype}/{w.y_dtype}",
                   "name": w.name, "n_tokens": B, "hidden": w.hidden, "depth": w.depth, "n_trees": w.n_trees,
                   "layers": NL, "norm": bool(args.norm), "mode": args.mode, "plan": plan},
        "kernel_us": {"mean": t["mean_ms"] * 1e3, "min": t["min_ms"] * 1e3, "std": t["std_ms"] * 1e3},
        "timing": f"value and ms_per_step: the {args.steps} timed steps back to back between one pair of HIP "
                  f"events on the launch stream; kernel_us and roofline: a second pass of {args.steps} steps, each "
                  f"between its own pair of events",
    }

    # Measured HBM bytes per launch from a committed counter summary, valid only while the
    # kernel sources are the ones the counters were taken on.
    from paper_2311_10770_amd.rocprof_summary import kernel_source_hash

    traffic = None
    tname = f"traffic_{w.name}_{args.mode}{'_backward' if args.backward else ''}.json"
    tpath = Path(args.traffic) if args.traffic else ROOT / "profiles" / tname
    if tpath.exists():
        summ = json.loads(tpath.read_text())
        if summ.get("kernel_source_hash") == kernel_source_hash(args.backward):
            traffic = summ.get("hbm_bytes_per_launch")
        else:
            log(f"{tpath.name} was taken on other kernel sources: traffic unreported")
    if "grouped<" in plan:
        kernels = "walk_kernel + emit_kernel"
    elif "tiled<" in plan:
        kernels = "fill_i32_kernel + walk_kernel + tile_kernel"
    else:
        kernels = plan.split("<")[0].split()[-1] + "_kernel"
    if plan.startswith("per-layer"):
        kernels = f"{NL} launches of {kernels}"
    if args.backward:
        # compulsory HBM bytes of one backward: x, dy and dx rows, the forward's records (logits and
        # leaf per token and tree), both weight matrices read and both fp32 dW matrices written
        sz = {"bf16": 2, "f32": 4}
        per_tok = w.hidden * (2 * sz[w.x_dtype] + sz[w.y_dtype]) + 4 * w.n_trees * (w.depth + 2)
        bwd_bytes = B * per_tok + w.n_trees * w.nodes * w.hidden * 2 * (sz[w.w_dtype] + 4)
        kernels = ("bwd_rank_wave_kernel + bwd_leafsum_kernel + bwd_base_kernel (+ bwd_scan_kernel past 4096 "
                   "leaves) + bwd_place_kernel + bwd_fused_kernel + bwd_wsum_kernel" if fused else
                   "bwd_token_kernel + sort kernels + bwd_wtile_kernel / bwd_piece_kernel + fix-up")
        bach = bwd_bytes / (ms / 1e3) / 1e9
        out["roofline"] = {"bound": "hbm", "achieved": bach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                           "frac": bach / HBM_PEAK_GBS, "traffic": traffic, "kernels": kernels,
                           "basis": f"compulsory bytes of one backward = {B} tokens x {per_tok} B (x, dy, dx rows, "
                                    f"logits and leaf) + {w.n_trees * w.nodes * w.hidden * 2 * (sz[w.w_dtype] + 4)} B "
                                    f"(W read, fp32 dW written), over the mean backward time of the timed region "
                                    f"(ms_per_step: back to back between one pair of HIP events on the launch "
                                    f"stream; {kernels})"}
    else:
        C = w.compulsory_bytes(B) * NL
        cach = C / (ms / 1e3) / 1e9
        out["roofline"] = {"bound": "hbm", "achieved": cach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                           "frac": cach / HBM_PEAK_GBS, "traffic": traffic, "kernels": kernels,
                           "algorithmic_bytes": C,
                           "traffic_over_algorithmic": (traffic / C) if traffic else None,
                           "basis": f"compulsory HBM bytes of one forward C = B H (s_x + s_y) + T 2 H s_w "
                                    f"sum_l 2^l (1 - (1 - 2^-l)^B) = {C / 1e6:.1f} MB ({NL} layer(s): x read once, y "
                                    f"written once, every weight row the batch touches read once), over the mean "
                                    f"forward time of the timed region (ms_per_step: {args.steps} forwards back to "
                                    f"back between one pair of HIP events on the launch stream; {kernels})"}
        out["gathered"] = {"bytes_per_forward": gathered, "gbs": gathered / (ms / 1e3) / 1e9,
                           "over_hbm_peak": gathered / (ms / 1e3) / 1e9 / HBM_PEAK_GBS,
                           "per_call_gbs": achieved,
                           "basis": f"{w.gathered_bytes_per_token()} B per token (one W_in and one W_out row per "
                                    f"visited node) x {B} tokens x {NL} layer(s), over ms_per_step (per_call_gbs: "
                                    f"over the mean of calls each between their own events); served mostly by "
                                    f"LDS, L2 and MALL, not HBM"}
    if args.cold_reps:
        tc = benchlib.time_cold(step, args.cold_reps, stream)
        out["cold"] = {"kernel_us": {"mean": tc["mean_ms"] * 1e3, "min": tc["min_ms"] * 1e3,
                                     "std": tc["std_ms"] * 1e3},
                       "tokens_per_s": B / (tc["mean_ms"] / 1e3),
                       "timing": f"{args.cold_reps} calls, each after a 1 GiB write that evicts the weights from "
                                 f"L2 and MALL, each between its own pair of HIP events"}
        log(f"cold: {tc['mean_ms'] * 1e3:.1f} us per call (warm {t['mean_ms'] * 1e3:.1f})")
    flops = w.flops_per_token() * B * NL * (2 if args.backward else 1)  # backward: dot + axpy + two row updates
    out["alu"] = {"achieved_tflops": flops / (t["mean_ms"] / 1e3) / 1e12, "peak_tflops_fp32_vector": 157.3}

    if NL > 1:
        # the persistent stack kernel (mode descent) beside the planned step
        kd = dict(kw, mode="descent")
        tk = benchlib.time_launches(lambda: fff.forward_stack(x, dlayers, w.depth, w.n_trees, y, **kd),
                                    max(10, args.steps // 4), 3, stream)
        out["stack"] = {"persistent_kernel_ms": tk["mean_ms"], "step_ms": t["mean_ms"],
                        "persistent_plan": fff.describe_stack(x, dlayers, w.depth, w.n_trees, y, **kd)}
        log(f"persistent stack kernel: {tk['mean_ms'] * 1e3:.1f} us vs the planned step {t['mean_ms'] * 1e3:.1f} us")

    if not args.backward and not args.no_valu_only and NL == 1 and ("tiled<" in plan or "masked<" in plan):
        # the same layer without matrix cores: the grouped walk + emit (one tree) or the fused kernel
        vmode = "grouped" if w.n_trees == 1 and w.depth >= 3 else "descent"
        vkw = dict(kw, mode=vmode)
        tv = benchlib.time_launches(lambda: fff.forward(x, wi, wo, w.depth, w.n_trees, y, **vkw, **layer_kw(0)),
                                    args.steps, args.warmup, stream)
        vms = tv["region_ms"] / args.steps
        out["valu_only"] = {"mode": vmode, "ms_per_step": vms, "tokens_per_s": B / (vms / 1e3),
                            "roofline_frac": w.compulsory_bytes(B) / (vms / 1e3) / 1e9 / HBM_PEAK_GBS,
                            "plan": fff.describe(x, wi, wo, w.depth, w.n_trees, y, **vkw, **layer_kw(0)),
                            "why": "the default plan accumulates the outputs of tokens that share a leaf on "
                                   "MFMA; this is the layer on the vector ALU alone"}
        log(f"vector-ALU plan ({vmode}): {vms * 1e3:.1f} us/step, {B / (vms / 1e3) / 1e6:.1f} M tok/s")

    if not args.no_dense and not args.backward:
        H, F = w.hidden, 3072 if w.hidden == 768 else 4 * w.hidden
        g = torch.Generator(device="cpu").manual_seed(1234)
        w1_f = torch.randn(F, H, generator=g) / H ** 0.5
        w2_f = torch.randn(H, F, generator=g) / F ** 0.5
        out["dense"] = {}
        dtypes = ["bf16"] + (["f32"] if w.x_dtype == "f32" else [])
        for ddt in dtypes:
            tdt = torch.bfloat16 if ddt == "bf16" else torch.float32
            w1, w2 = w1_f.to(dev, tdt), w2_f.to(dev, tdt)
            xb = x if x.dtype == tdt else x.to(tdt)
            dense = benchlib.DenseFF(xb, w1, w2)

            def dense_step():  # one dense layer per FFF layer of the workload
                for _ in range(NL):
                    dense()

            nd = max(20, args.steps // 2)
            td = benchlib.time_launches(dense_step, nd, 10, stream)
            dense_ms = td["region_ms"] / nd
            # sanity: the fused-epilogue GEMMs compute the dense layer (tanh- vs erf-GELU differ slightly)
            ref = torch.nn.functional.linear(torch.nn.functional.gelu(torch.nn.functional.linear(
                xb[:1024].float(), w1.float())), w2.float())
            rel = float((dense.y[:1024].float() - ref).norm() / ref.norm())
            dflops = dense.flops * NL
            peak = MFMA_PEAK_TFLOPS[ddt]
            ach = dflops / (dense_ms / 1e3) / 1e12
            d = {"what": f"{NL} x " * (NL > 1) + f"dense FF {H}->{F}->{H} on the same tokens, {ddt}: {dense.info}",
                 "ms": dense_ms, "tokens_per_s": B / (dense_ms / 1e3), "speedup_fff_over_dense": dense_ms / ms,
                 "flops": dflops, "achieved_tflops": ach, "mfma_peak_tflops": peak, "frac_of_mfma_peak": ach / peak,
                 "speedup_fff_over_dense_at_mfma_peak": (dflops / (peak * 1e12) * 1e3) / ms,
                 "rel_err_vs_fp32_torch": rel}
            if "valu_only" in out:
                d["speedup_valu_only_over_dense"] = dense_ms / out["valu_only"]["ms_per_step"]
            if ddt == "bf16":
                def dense_unfused():
                    for _ in range(NL):
                        torch.nn.functional.linear(torch.nn.functional.gelu(torch.nn.functional.linear(xb, w1)), w2)

                tu = benchlib.time_launches(dense_unfused, nd, 5, stream)
                d["torch_unfused_ms"] = tu["region_ms"] / nd
                d["speedup_fff_over_torch_unfused"] = d["torch_unfused_ms"] / ms
            if args.cold_reps and ddt == "bf16":
                tdc = benchlib.time_cold(dense_step, args.cold_reps, stream)
                d["cold_ms"] = tdc["mean_ms"]
                d["speedup_fff_over_dense_cold"] = tdc["mean_ms"] / out["cold"]["kernel_us"]["mean"] * 1e3
            dense.close()
            out["dense"][ddt] = d
            log(f"dense {ddt} (hipBLASLt, fused GELU): {dense_ms * 1e3:.1f} us/step ({ach:.0f} TFLOP/s, "
                f"{ach / peak:.0%} of the MFMA peak) -> speedup {dense_ms / ms:.2f}x, "
                f"{d['speedup_fff_over_dense_at_mfma_peak']:.2f}x against a dense layer at peak (rel err {rel:.1e})")
        # the headline comparison: the dense layer in the workload's weight type
        out["dense"]["speedup_fff_over_dense"] = out["dense"]["f32" if w.w_dtype == "f32" else "bf16"][
            "speedup_fff_over_dense"]
        out["paper"] = PAPER_SPEEDUPS

    if args.backward:
        args.no_cpu_baseline = True  # the backward's CPU leg and check live in the tests

    if not args.no_cpu_baseline:
        # The CPU leg: the fp64 oracle timed on the host cores over the first n tokens.  Its
        # outputs for those tokens are also compared with the device's (after the timed region).
        import oracle
        from oracle import parity

        threads = oracle.default_threads()
        n = min(B, 4096 if NL == 1 else 1024)
        eps = kw.get("norm_eps")

        def cpu_pass(records):
            if NL == 1 and not args.norm:
                return oracle.forward(L["x"][:n], layers_np[0]["w_in"], layers_np[0]["w_out"], w.depth, w.n_trees,
                                      records=records, threads=threads)
            return oracle.stack(L["x"][:n], layers_np, w.depth, w.n_trees, w.y_dtype, norm_eps=eps, threads=threads)

        ref = cpu_pass(True)
        done, t0 = 0, time.perf_counter()
        while True:
            cpu_pass(False)
            done += n
            if time.perf_counter() - t0 >= args.cpu_seconds:
                break
        el = time.perf_counter() - t0
        # the same oracle on one thread over a tenth of the sample, for the per-core rate
        n1 = max(1, n // 10)
        t1 = time.perf_counter()
        if NL == 1 and not args.norm:
            oracle.forward(L["x"][:n1], layers_np[0]["w_in"], layers_np[0]["w_out"], w.depth, w.n_trees,
                           records=False, threads=1)
        else:
            oracle.stack(L["x"][:n1], layers_np, w.depth, w.n_trees, w.y_dtype, norm_eps=eps, threads=1)
        el1 = time.perf_counter() - t1
        out["cpu_baseline"] = {"value": done / el, "unit": "tokens/s", "cores": threads, "kind": "oracle",
                               "sample": f"first {n} tokens of the same batch, repeated {done // n}x over "
                                         f"{el:.1f}s wall, fp64 C oracle on {threads} host threads",
                               "single_thread_value": n1 / el1, "host": host_cpu()}
        log(f"cpu oracle: {done / el:.0f} tok/s on {threads} threads, {n1 / el1:.0f} on one")
        if not args.no_check:
            # the last layer, on the device's own input to it, against the oracle's block
            nodes = torch.empty((NL, B, w.n_trees, w.depth + 1), dtype=torch.int32, device=dev)
            x_last = x
            if NL > 1:
                prev = torch.empty_like(y)
                fff.forward_stack(x, dlayers[:-1], w.depth, w.n_trees, prev, mode=args.mode,
                                  lds_levels=args.lds_levels, **({} if not args.norm else
                                                                 dict(norm="layernorm", norm_eps=eps)))
                x_last = prev
            step()
            fff.forward(x_last, dlayers[-1][0], dlayers[-1][1], w.depth, w.n_trees, torch.empty_like(y),
                        nodes_out=nodes[-1], out="residual" if NL > 1 else "store", **kw, **layer_kw(NL - 1))
            torch.cuda.synchronize()
            xl = fff.to_numpy(x_last)[:n]
            lay = layers_np[-1]
            if NL == 1 and not args.norm:
                r = ref
                u, base = L["x"][:n], None
            else:
                r = oracle.block(xl, lay["w_in"], lay["w_out"], w.depth, w.n_trees,
                                 norm={"gamma": lay.get("gamma"), "beta": lay.get("beta"), "eps": eps}
                                 if args.norm else None, threads=threads)
                u, base = r["u"], (xl if NL > 1 else None)
                r = dict(r, y=r["fff"])
            rep = parity.check(u, lay["w_in"], lay["w_out"], w.depth, w.n_trees, r, fff.to_numpy(y)[:n],
                               nodes[-1].cpu().numpy()[:n], tol=2e-2 if w.y_dtype == "bf16" else 1e-5, base_dev=base)
            out["cpu_baseline"]["check"] = {"tokens": n, "layer_checked": NL - 1, "ok": rep["ok"],
                                            "max_normwise_err_raw": rep["max_normwise_err_raw"],
                                            "n_conditioned": rep["n_conditioned"],
                                            "n_ill_conditioned": rep["n_ill_conditioned"],
                                            "bf16_elem_excess": rep.get("bf16_elem_excess"),
                                            "n_near_tie": rep["n_near_tie"],
                                            "n_path_divergent": rep["n_path_divergent"]}
            log("device vs oracle on the sample:", out["cpu_baseline"]["check"])

    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
