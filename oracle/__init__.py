"""fp64 CPU oracle for FFF inference -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, the smoke check in ``__graft_entry__`` and the benchmark's
CPU-baseline leg may import this package.  It shares no code with the HIP
path (``paper_2311_10770_amd``) and neither imports the other.

The arithmetic lives in ``fff_oracle.c`` (plain C, fp64, built with gcc into
``liboracle.so``); this module only marshals numpy arrays.  Inputs are numpy
arrays: float32, or uint16 holding bf16 bit patterns (the FFF input may also
be float64, e.g. the output of ``layer_norm``, and so may the weights of
the finite-difference pins).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from pathlib import Path

import numpy as np

_HERE = Path(__file__).resolve().parent
_SRC = _HERE / "fff_oracle.c"
_LIB = _HERE / "liboracle.so"

ACT_GELU_ERF, ACT_GELU_TANH, ACT_IDENTITY = 0, 1, 2
_ACTS = {"gelu": ACT_GELU_ERF, "gelu_erf": ACT_GELU_ERF, "gelu_tanh": ACT_GELU_TANH,
         "identity": ACT_IDENTITY}
DEFAULT_TIE_REL = 1e-5

_lib = None


def build(force: bool = True) -> Path:
    """Compile liboracle.so with gcc (plain -O2, no fast-math, no FMA contraction)."""
    if force or not _LIB.exists():
        tmp = _LIB.with_suffix(".so.tmp")
        cmd = ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-pthread", "-ffp-contract=off",
               "-fno-fast-math", "-Wall", "-Wextra", "-o", str(tmp), str(_SRC), "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not _LIB.exists():
        build(force=False)
    lib = ctypes.CDLL(str(_LIB))
    vp, i32, i64, dbl = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.oracle_activation.argtypes = [dbl, ctypes.c_int]
    lib.oracle_activation.restype = dbl
    lib.oracle_forward.argtypes = [vp, ctypes.c_int, vp, vp, ctypes.c_int, i64, i32, i32, i32,
                                   ctypes.c_int, dbl, vp, vp, vp, vp, ctypes.c_int]
    lib.oracle_forward.restype = ctypes.c_int
    lib.oracle_eval_path.argtypes = [vp, ctypes.c_int, vp, vp, ctypes.c_int, i32, i32, i32,
                                     ctypes.c_int, vp, vp, vp]
    lib.oracle_eval_path.restype = ctypes.c_int
    lib.oracle_layer_norm.argtypes = [vp, ctypes.c_int, i64, i32, vp, vp, dbl, vp]
    lib.oracle_layer_norm.restype = ctypes.c_int
    lib.oracle_round_bf16.argtypes = [vp, i64, vp]
    lib.oracle_round_bf16.restype = ctypes.c_int
    lib.oracle_activation_grad.argtypes = [dbl, ctypes.c_int]
    lib.oracle_activation_grad.restype = dbl
    lib.oracle_backward.argtypes = [vp, ctypes.c_int, vp, vp, ctypes.c_int, vp, vp, i64, i32, i32, i32,
                                    ctypes.c_int, vp, vp, vp]
    lib.oracle_backward.restype = ctypes.c_int
    _lib = lib
    return lib


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return 0
    if a.dtype == np.uint16:
        return 1
    if a.dtype == np.float64:
        return 2
    raise TypeError(f"oracle inputs must be float32, float64 or uint16 (bf16 bits), got {a.dtype}")


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _act(act) -> int:
    return _ACTS[act] if isinstance(act, str) else int(act)


def activation(z: float, act="gelu") -> float:
    return _load().oracle_activation(float(z), _act(act))


def activation_grad(z: float, act="gelu") -> float:
    return _load().oracle_activation_grad(float(z), _act(act))


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return max(1, os.cpu_count() or 1)


def forward(x: np.ndarray, w_in: np.ndarray, w_out: np.ndarray, depth: int, n_trees: int,
            act="gelu", tie_rel: float = DEFAULT_TIE_REL, records: bool = True,
            threads: int | None = None) -> dict:
    """FFF forward in fp64.

    Returns ``{"y": [B,H] float64}`` and, if ``records``, also ``nodes``
    (int32), ``logits`` (float64) and ``near_tie`` (bool), each [B, T, D+1].
    """
    x = np.ascontiguousarray(x)
    w_in = np.ascontiguousarray(w_in)
    w_out = np.ascontiguousarray(w_out)
    if w_in.dtype != w_out.dtype:
        raise TypeError("W_in and W_out must share a dtype")
    B, H = x.shape
    N = (1 << (depth + 1)) - 1
    if w_in.shape != (n_trees, N, H) or w_out.shape != (n_trees, N, H):
        raise ValueError(f"weights must be [{n_trees}, {N}, {H}], got {w_in.shape}, {w_out.shape}")
    y = np.empty((B, H), dtype=np.float64)
    nodes = logits = tie = None
    if records:
        nodes = np.empty((B, n_trees, depth + 1), dtype=np.int32)
        logits = np.empty((B, n_trees, depth + 1), dtype=np.float64)
        tie = np.empty((B, n_trees, depth + 1), dtype=np.uint8)
    rc = _load().oracle_forward(_ptr(x), _dtype_code(x), _ptr(w_in), _ptr(w_out), _dtype_code(w_in),
                                B, H, depth, n_trees, _act(act), float(tie_rel), _ptr(y), _ptr(nodes),
                                _ptr(logits), _ptr(tie), int(threads or default_threads()))
    if rc != 0:
        raise RuntimeError(f"oracle_forward failed with {rc}")
    out = {"y": y}
    if records:
        out.update(nodes=nodes, logits=logits, near_tie=tie.astype(bool))
    return out


def eval_path(x_row: np.ndarray, w_in: np.ndarray, w_out: np.ndarray, depth: int, n_trees: int,
              path: np.ndarray, act="gelu") -> tuple[np.ndarray, np.ndarray]:
    """fp64 output and logits of ONE token along a given path [T, D+1]."""
    x_row = np.ascontiguousarray(x_row).reshape(-1)
    w_in = np.ascontiguousarray(w_in)
    w_out = np.ascontiguousarray(w_out)
    path = np.ascontiguousarray(path, dtype=np.int32).reshape(n_trees, depth + 1)
    H = x_row.shape[0]
    y = np.empty(H, dtype=np.float64)
    logits = np.empty((n_trees, depth + 1), dtype=np.float64)
    rc = _load().oracle_eval_path(_ptr(x_row), _dtype_code(x_row), _ptr(w_in), _ptr(w_out),
                                  _dtype_code(w_in), H, depth, n_trees, _act(act), _ptr(path), _ptr(y),
                                  _ptr(logits))
    if rc == -3:
        raise ValueError("path is not a root-to-leaf walk")
    if rc != 0:
        raise RuntimeError(f"oracle_eval_path failed with {rc}")
    return y, logits


def _widen(a: np.ndarray) -> np.ndarray:
    """Exact float64 value of a float32 / float64 / bf16-bits array."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def layer_norm(x: np.ndarray, gamma=None, beta=None, eps: float = 1e-12) -> np.ndarray:
    """Row-wise LayerNorm of x [B,H] in fp64 (biased variance, eps inside the root)."""
    x = np.ascontiguousarray(x)
    B, H = x.shape
    g = None if gamma is None else np.ascontiguousarray(_widen(gamma).reshape(H))
    b = None if beta is None else np.ascontiguousarray(_widen(beta).reshape(H))
    out = np.empty((B, H), dtype=np.float64)
    rc = _load().oracle_layer_norm(_ptr(x), _dtype_code(x), B, H, _ptr(g), _ptr(b), float(eps), _ptr(out))
    if rc != 0:
        raise RuntimeError(f"oracle_layer_norm failed with {rc}")
    return out


def round_bf16(v: np.ndarray) -> np.ndarray:
    """Nearest bf16 (ties to even) of float64 values, as uint16 bit patterns."""
    v = np.ascontiguousarray(v, dtype=np.float64)
    out = np.empty(v.shape, dtype=np.uint16)
    rc = _load().oracle_round_bf16(_ptr(v), v.size, _ptr(out))
    if rc != 0:
        raise RuntimeError(f"oracle_round_bf16 failed with {rc}")
    return out


def store_as(v: np.ndarray, dtype: str) -> np.ndarray:
    """A float64 result stored in a device dtype: float32 (nearest) or bf16 bits (nearest even)."""
    return round_bf16(v) if dtype == "bf16" else v.astype(np.float32)


def block(x: np.ndarray, w_in: np.ndarray, w_out: np.ndarray, depth: int, n_trees: int, norm=None,
          act="gelu", tie_rel: float = DEFAULT_TIE_REL, threads: int | None = None) -> dict:
    """The intermediate layer of a pre-norm block, x + FFF(norm(x)), in fp64.

    ``norm``: None (FFF of x itself) or a dict with ``gamma``, ``beta`` (arrays or
    None) and ``eps``: LayerNorm first.  Returns ``forward``'s dict for the FFF
    input ``u`` (also returned), with ``y`` replaced by x + FFF(u) and the bare
    FFF output kept as ``fff``.
    """
    u = x if norm is None else layer_norm(x, norm.get("gamma"), norm.get("beta"), norm["eps"])
    out = forward(u, w_in, w_out, depth, n_trees, act=act, tie_rel=tie_rel, threads=threads)
    out["fff"] = out["y"]
    out["y"] = _widen(x) + out["fff"]
    out["u"] = _widen(u)
    return out


def stack(x: np.ndarray, layers, depth: int, n_trees: int, store_dtype: str, norm_eps=None, act="gelu",
          threads: int | None = None) -> list:
    """Layers x_{i+1} = store(x_i + FFF_i(norm_i(x_i))), each result stored in ``store_dtype``.

    ``layers``: a list of dicts with ``w_in``, ``w_out`` and, when ``norm_eps`` is
    not None, optional ``gamma`` / ``beta``.  Returns the per-layer ``block``
    dicts, each with ``x_in`` (the stored input) and ``x_out`` (the stored output).
    """
    outs = []
    for lay in layers:
        norm = None if norm_eps is None else {"gamma": lay.get("gamma"), "beta": lay.get("beta"), "eps": norm_eps}
        r = block(x, lay["w_in"], lay["w_out"], depth, n_trees, norm=norm, act=act, threads=threads)
        r["x_in"] = x
        x = store_as(r["y"], store_dtype)
        r["x_out"] = x
        outs.append(r)
    return outs


def backward(x: np.ndarray, w_in: np.ndarray, w_out: np.ndarray, depth: int, n_trees: int, dy: np.ndarray,
             path: np.ndarray, act="gelu") -> dict:
    """Hard-routed backward in fp64 along the given paths [B, T, D+1].

    Returns ``dx`` [B,H], ``dw_in`` and ``dw_out`` [T,N,H] (float64; rows off
    every path are zero)."""
    x = np.ascontiguousarray(x)
    w_in = np.ascontiguousarray(w_in)
    w_out = np.ascontiguousarray(w_out)
    B, H = x.shape
    N = (1 << (depth + 1)) - 1
    if w_in.shape != (n_trees, N, H) or w_out.shape != (n_trees, N, H) or w_in.dtype != w_out.dtype:
        raise ValueError("weights must be [T, N, H] of one dtype")
    dy = np.ascontiguousarray(_widen(dy).reshape(B, H))
    path = np.ascontiguousarray(path, dtype=np.int32).reshape(B, n_trees, depth + 1)
    dx = np.empty((B, H))
    dwi = np.empty((n_trees, N, H))
    dwo = np.empty((n_trees, N, H))
    rc = _load().oracle_backward(_ptr(x), _dtype_code(x), _ptr(w_in), _ptr(w_out), _dtype_code(w_in), _ptr(dy),
                                 _ptr(path), B, H, depth, n_trees, _act(act), _ptr(dx), _ptr(dwi), _ptr(dwo))
    if rc == -3:
        raise ValueError("a path is not a root-to-leaf walk")
    if rc != 0:
        raise RuntimeError(f"oracle_backward failed with {rc}")
    return {"dx": dx, "dw_in": dwi, "dw_out": dwo}
