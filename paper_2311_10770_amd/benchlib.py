"""ctypes binding of libfffbench.so: the hipBLASLt dense feedforward comparator
and the copy kernel used to calibrate HBM counters.  Benchmark-only."""
from __future__ import annotations

import ctypes
import time
from ctypes import c_double, c_char_p, c_int, c_int32, c_int64, c_void_p
from pathlib import Path

import torch

LIB_PATH = Path(__file__).resolve().with_name("libfffbench.so")
_lib = None


def load():
    global _lib
    if _lib is None:
        if not LIB_PATH.exists():
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2311_10770_amd.build`")
        lib = ctypes.CDLL(str(LIB_PATH))
        lib.fffb_dense_ff_create.argtypes = [c_int64, c_int32, c_int32, c_int32, c_void_p, c_void_p, c_void_p,
                                             c_void_p, c_void_p, c_void_p]
        lib.fffb_dense_ff_create.restype = c_void_p
        lib.fffb_dense_ff_info.argtypes = [c_void_p]
        lib.fffb_dense_ff_info.restype = c_char_p
        lib.fffb_dense_ff_run.argtypes = [c_void_p] * 6 + [c_void_p]
        lib.fffb_dense_ff_run.restype = c_int
        lib.fffb_dense_ff_destroy.argtypes = [c_void_p]
        lib.fffb_dense_ff_destroy.restype = None
        lib.fffb_copy.argtypes = [c_void_p, c_void_p, c_int64, c_void_p]
        lib.fffb_copy.restype = c_int
        lib.fffb_mb_read.argtypes = [c_void_p, c_int64, c_int64, c_void_p, c_int, c_void_p]
        lib.fffb_mb_read.restype = c_int
        lib.fffb_mb_write.argtypes = [c_void_p, c_int64, c_int64, c_int, c_void_p]
        lib.fffb_mb_write.restype = c_int
        lib.fffb_mb_gather.argtypes = [c_void_p, c_int64, c_int, c_int, c_int, c_int, c_void_p, c_void_p]
        lib.fffb_mb_gather.restype = c_int
        lib.fffb_mb_mfma.argtypes = [c_int, c_int, c_int, c_int, c_void_p, c_void_p]
        lib.fffb_mb_mfma.restype = c_double
        _lib = lib
    return _lib


class DenseFF:
    """y = GELU(x W1^T) W2^T on hipBLASLt (x, W1 and W2 all bf16 or all fp32; fp32 accumulation),
    GELU fused in the first GEMM's epilogue."""

    def __init__(self, x: torch.Tensor, w1: torch.Tensor, w2: torch.Tensor, stream=None):
        lib = load()
        if not (x.dtype == w1.dtype == w2.dtype) or x.dtype not in (torch.bfloat16, torch.float32):
            raise ValueError("x, W1 and W2 must all be bf16 or all fp32")
        self.x, self.w1, self.w2 = x, w1, w2
        B, H = x.shape
        F = w1.shape[0]
        self.flops = 4 * B * H * F
        self.h = torch.empty((B, F), dtype=x.dtype, device=x.device)
        self.y = torch.empty((B, H), dtype=x.dtype, device=x.device)
        self.stream = (stream or torch.cuda.current_stream(x.device)).cuda_stream
        self.handle = lib.fffb_dense_ff_create(B, H, F, int(x.dtype == torch.float32), x.data_ptr(), w1.data_ptr(),
                                               w2.data_ptr(), self.h.data_ptr(), self.y.data_ptr(), self.stream)
        if not self.handle:
            raise RuntimeError("hipBLASLt dense FF setup failed")
        self.info = lib.fffb_dense_ff_info(self.handle).decode()

    def __call__(self):
        rc = load().fffb_dense_ff_run(self.handle, self.x.data_ptr(), self.w1.data_ptr(), self.w2.data_ptr(),
                                      self.h.data_ptr(), self.y.data_ptr(), self.stream)
        if rc != 0:
            raise RuntimeError(f"hipBLASLt matmul failed ({rc})")
        return self.y

    def close(self):
        if self.handle:
            load().fffb_dense_ff_destroy(self.handle)
            self.handle = None


def copy(src: torch.Tensor, dst: torch.Tensor, stream=None):
    s = (stream or torch.cuda.current_stream(src.device)).cuda_stream
    rc = load().fffb_copy(src.data_ptr(), dst.data_ptr(), src.numel() * src.element_size(), s)
    if rc != 0:
        raise RuntimeError(f"fffb_copy failed ({rc})")


def time_launches(fn, steps: int, warmup: int, stream):
    """Two timed passes of `steps` calls on `stream` after `warmup` untimed ones.

    region_ms: the first pass, the calls back to back between one pair of events
    (a timing event between every call would leave the GPU idle for a few
    microseconds per call; a serving loop has none).  mean/min/max/std_ms: the
    second pass, every call between its own pair of events: the duration of one
    call's kernels."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(steps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    region_ms = e0.elapsed_time(e1)
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    for i in range(steps):
        starts[i].record(stream)
        fn()
        ends[i].record(stream)
    torch.cuda.synchronize()
    per = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    return {"mean_ms": sum(per) / steps, "min_ms": min(per), "max_ms": max(per),
            "std_ms": (sum((p - sum(per) / steps) ** 2 for p in per) / steps) ** 0.5,
            "region_ms": region_ms, "wall_s": wall}


def time_cold(fn, reps: int, stream, flush_bytes: int = 1 << 30):
    """Cold-cache timing: before each call a `flush_bytes` write (1 GiB: more than the 256 MB
    MALL and the eight 4 MB L2s together) evicts the weights; only the call sits between its
    pair of events on `stream`.  Returns mean/min/std_ms over `reps` calls."""
    scratch = torch.empty(flush_bytes, dtype=torch.uint8, device=torch.device("cuda", torch.cuda.current_device()))
    fn()
    torch.cuda.synchronize()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(reps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(reps)]
    with torch.cuda.stream(stream):
        for i in range(reps):
            scratch.fill_(i & 0xFF)
            starts[i].record(stream)
            fn()
            ends[i].record(stream)
    torch.cuda.synchronize()
    per = [a.elapsed_time(b) for a, b in zip(starts, ends)]
    mean = sum(per) / reps
    del scratch
    return {"mean_ms": mean, "min_ms": min(per), "std_ms": (sum((q - mean) ** 2 for q in per) / reps) ** 0.5}
