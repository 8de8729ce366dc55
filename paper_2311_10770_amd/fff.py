"""ctypes binding of libfff.so (include/fff.h).

Argument marshalling only: tensors become device pointers, enums become
ints, and every step of the FFF forward runs in the library's HIP kernels.
The library must be built (``python -m paper_2311_10770_amd.build``); there
is no fallback path, and a missing library raises.
"""
from __future__ import annotations

import ctypes
from ctypes import c_char_p, c_int, c_int32, c_int64, c_size_t, c_void_p
from pathlib import Path

import torch

LIB_PATH = Path(__file__).resolve().with_name("libfff.so")

FFF_OK, FFF_ERR_INVALID_ARG, FFF_ERR_UNSUPPORTED, FFF_ERR_WORKSPACE, FFF_ERR_HIP = 0, -1, -2, -3, -4
FFF_F32, FFF_BF16 = 0, 1
ACTS = {"gelu": 0, "gelu_erf": 0, "gelu_tanh": 1, "identity": 2}
MODES = {"auto": 0, "descent": 1, "grouped": 2, "generic": 3, "tiled": 4, "masked": 5, "subtree": 6}
OUTS = {"store": 0, "accumulate": 1, "residual": 2}
NORMS = {None: 0, "none": 0, "layernorm": 1}
_TORCH_DT = {torch.float32: FFF_F32, torch.bfloat16: FFF_BF16}


class FffArgs(ctypes.Structure):
    """Mirror of ``fff_args`` in include/fff.h."""

    _fields_ = [
        ("x", c_void_p), ("W_in", c_void_p), ("W_out", c_void_p), ("y", c_void_p),
        ("n_tokens", c_int64), ("hidden", c_int32), ("depth", c_int32), ("n_trees", c_int32),
        ("x_dtype", c_int32), ("w_dtype", c_int32), ("y_dtype", c_int32),
        ("act", c_int32), ("mode", c_int32), ("out_mode", c_int32),
        ("lds_levels", c_int32), ("split_level", c_int32),
        ("nodes_out", c_void_p), ("logits_out", c_void_p),
        ("workspace", c_void_p), ("workspace_bytes", c_size_t),
        ("hip_stream", c_void_p),
        ("norm", c_int32), ("norm_eps", ctypes.c_float), ("norm_gamma", c_void_p), ("norm_beta", c_void_p),
    ]


class FffLayer(ctypes.Structure):
    """Mirror of ``fff_layer`` in include/fff.h."""

    _fields_ = [("W_in", c_void_p), ("W_out", c_void_p), ("norm_gamma", c_void_p), ("norm_beta", c_void_p)]


class FffBackwardArgs(ctypes.Structure):
    """Mirror of ``fff_backward_args`` in include/fff.h."""

    _fields_ = [
        ("x", c_void_p), ("W_in", c_void_p), ("W_out", c_void_p), ("dy", c_void_p),
        ("leaves", c_void_p), ("logits", c_void_p),
        ("dx", c_void_p), ("dW_in", c_void_p), ("dW_out", c_void_p),
        ("n_tokens", c_int64), ("hidden", c_int32), ("depth", c_int32), ("n_trees", c_int32),
        ("x_dtype", c_int32), ("w_dtype", c_int32), ("dy_dtype", c_int32), ("dx_dtype", c_int32),
        ("act", c_int32), ("accumulate", c_int32), ("bad_leaves", c_void_p),
        ("workspace", c_void_p), ("workspace_bytes", c_size_t), ("hip_stream", c_void_p),
    ]


class FffError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(msg)
        self.status = status


_lib = None

EXPORTS = ("fff_forward", "fff_forward_ex", "fff_forward_static", "fff_workspace_bytes", "fff_describe", "fff_forward_stack",
           "fff_describe_stack", "fff_backward", "fff_backward_workspace_bytes", "fff_status_str",
           "fff_last_hip_error", "fff_version")


def load_library(path: Path | str | None = None):
    """Load libfff.so once; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    p = Path(path) if path else LIB_PATH
    if not p.exists():
        raise RuntimeError(f"{p} is missing: build it with `python -m paper_2311_10770_amd.build`")
    lib = ctypes.CDLL(str(p))
    lib.fff_forward.argtypes = [c_void_p, c_void_p, c_void_p, c_int32, c_int32, c_void_p, c_int64, c_int32,
                                c_int32, c_int32, c_int32, c_void_p]
    lib.fff_forward.restype = c_int
    lib.fff_forward_ex.argtypes = [ctypes.POINTER(FffArgs)]
    lib.fff_forward_ex.restype = c_int
    lib.fff_forward_static.argtypes = [ctypes.POINTER(FffArgs)]
    lib.fff_forward_static.restype = c_int
    lib.fff_workspace_bytes.argtypes = [c_int64, c_int32, c_int32, c_int32, c_int32]
    lib.fff_workspace_bytes.restype = c_size_t
    lib.fff_describe.argtypes = [ctypes.POINTER(FffArgs), c_char_p, c_size_t]
    lib.fff_describe.restype = c_int
    lib.fff_forward_stack.argtypes = [ctypes.POINTER(FffArgs), ctypes.POINTER(FffLayer), c_int32]
    lib.fff_forward_stack.restype = c_int
    lib.fff_describe_stack.argtypes = [ctypes.POINTER(FffArgs), ctypes.POINTER(FffLayer), c_int32, c_char_p,
                                       c_size_t]
    lib.fff_describe_stack.restype = c_int
    lib.fff_backward.argtypes = [ctypes.POINTER(FffBackwardArgs)]
    lib.fff_backward.restype = c_int
    lib.fff_backward_workspace_bytes.argtypes = [c_int64, c_int32, c_int32, c_int32]
    lib.fff_backward_workspace_bytes.restype = c_size_t
    lib.fff_status_str.argtypes = [c_int]
    lib.fff_status_str.restype = c_char_p
    lib.fff_last_hip_error.argtypes = []
    lib.fff_last_hip_error.restype = c_int
    lib.fff_version.argtypes = []
    lib.fff_version.restype = c_int
    _lib = lib
    return lib


def status_str(rc: int) -> str:
    return load_library().fff_status_str(rc).decode()


def _check(rc: int):
    if rc != FFF_OK:
        lib = load_library()
        msg = status_str(rc)
        if rc == FFF_ERR_HIP:
            msg += f" (hipError {lib.fff_last_hip_error()})"
        raise FffError(rc, msg)


def _raw_stream(device: torch.device, stream=None) -> int:
    """The HIP stream handle a call is enqueued on: ``stream``'s, else the device's current one."""
    if stream is not None:
        return stream.cuda_stream
    getter = getattr(torch._C, "_cuda_getCurrentRawStream", None)
    if getter is not None:
        return getter(device.index if device.index is not None else torch.cuda.current_device())
    return torch.cuda.current_stream(device).cuda_stream


class _on_device:
    """``torch.cuda.device(device)`` when it is not already the current device (the library enqueues
    on the current device's stream and queries the current device's properties)."""

    def __init__(self, device: torch.device):
        self.ctx = None if device.index is None or device.index == torch.cuda.current_device() else \
            torch.cuda.device(device)

    def __enter__(self):
        if self.ctx is not None:
            self.ctx.__enter__()

    def __exit__(self, *exc):
        if self.ctx is not None:
            return self.ctx.__exit__(*exc)
        return False


def _dt(t: torch.Tensor, what: str) -> int:
    try:
        return _TORCH_DT[t.dtype]
    except KeyError:
        raise ValueError(f"{what} must be float32 or bfloat16, got {t.dtype}") from None


def _dev_tensor(t, what, device):
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{what} must be a torch.Tensor")
    if t.device != device:
        raise ValueError(f"{what} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    return t


def _check_weights(w_in, w_out, depth, n_trees, H, device):
    for t, what in ((w_in, "W_in"), (w_out, "W_out")):
        _dev_tensor(t, what, device)
    N = (1 << (depth + 1)) - 1
    if tuple(w_in.shape) != (n_trees, N, H) or tuple(w_out.shape) != (n_trees, N, H):
        raise ValueError(f"W_in/W_out must be [{n_trees}, {N}, {H}], got {tuple(w_in.shape)}, {tuple(w_out.shape)}")
    if w_in.dtype != w_out.dtype:
        raise ValueError("W_in and W_out must share a dtype")


def _check_norm_param(t, what, H, device):
    if t is None:
        return None
    _dev_tensor(t, what, device)
    if t.dtype != torch.float32 or t.numel() != H:
        raise ValueError(f"{what} must be a float32 tensor of {H} elements")
    return t.data_ptr()


def make_args(x, w_in, w_out, depth, n_trees, y, *, act="gelu", mode="auto", out="store", lds_levels=0,
              split_level=0, nodes_out=None, logits_out=None, workspace=None, stream=None, norm=None,
              norm_eps=1e-12, norm_gamma=None, norm_beta=None, n_layers=1) -> FffArgs:
    """Validate tensor-level properties and fill an ``fff_args``.  ``w_in`` / ``w_out`` may be None
    (stacks pass their weights per layer); records then hold ``n_layers`` layers."""
    if not isinstance(x, torch.Tensor) or x.dim() != 2:
        raise ValueError("x must be a 2-D tensor [n_tokens, hidden]")
    device = x.device
    if device.type != "cuda":
        raise ValueError("x must be a GPU tensor")
    _dev_tensor(y, "y", device)
    _dev_tensor(x, "x", device)
    B, H = x.shape
    if w_in is not None or w_out is not None:
        _check_weights(w_in, w_out, depth, n_trees, H, device)
    if tuple(y.shape) != (B, H):
        raise ValueError(f"y must be [{B}, {H}], got {tuple(y.shape)}")
    for t, what in ((nodes_out, "nodes_out"), (logits_out, "logits_out")):
        if t is not None:
            _dev_tensor(t, what, device)
            if t.numel() != n_layers * B * n_trees * (depth + 1):
                raise ValueError(f"{what} must hold n_layers*n_tokens*n_trees*(depth+1) elements")
    if nodes_out is not None and nodes_out.dtype != torch.int32:
        raise ValueError("nodes_out must be int32")
    if logits_out is not None and logits_out.dtype != torch.float32:
        raise ValueError("logits_out must be float32")
    a = FffArgs()
    a.x, a.y = x.data_ptr(), y.data_ptr()
    if w_in is not None:
        a.W_in, a.W_out = w_in.data_ptr(), w_out.data_ptr()
        a.w_dtype = _dt(w_in, "W_in")
    a.n_tokens, a.hidden, a.depth, a.n_trees = B, H, depth, n_trees
    a.x_dtype, a.y_dtype = _dt(x, "x"), _dt(y, "y")
    a.norm = NORMS[norm] if norm is None or isinstance(norm, str) else int(norm)
    a.norm_eps = float(norm_eps)
    a.norm_gamma = _check_norm_param(norm_gamma, "norm_gamma", H, device)
    a.norm_beta = _check_norm_param(norm_beta, "norm_beta", H, device)
    a.act = ACTS[act] if isinstance(act, str) else int(act)
    a.mode = MODES[mode] if isinstance(mode, str) else int(mode)
    a.out_mode = OUTS[out] if isinstance(out, str) else int(out)
    a.lds_levels, a.split_level = int(lds_levels), int(split_level)
    a.nodes_out = nodes_out.data_ptr() if nodes_out is not None else None
    a.logits_out = logits_out.data_ptr() if logits_out is not None else None
    if workspace is not None:
        _dev_tensor(workspace, "workspace", device)
        a.workspace, a.workspace_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    a.hip_stream = _raw_stream(device, stream)
    return a


_WORKSPACES: dict = {}
_NEED: dict = {}  # workspace bytes per (n_tokens, depth, n_trees, hidden)


def workspace_for(n_tokens: int, depth: int, n_trees: int, hidden: int, device, stream=None) -> torch.Tensor:
    """A cached device workspace large enough for every mode, one per (device, stream): calls on one
    stream run in order and share it; calls on different streams never share one.  A larger
    request replaces the stream's buffer (torch frees the old one in that stream's order)."""
    shape = (n_tokens, depth, n_trees, hidden)
    need = _NEED.get(shape)
    if need is None:
        need = _NEED[shape] = workspace_bytes(n_tokens, depth, n_trees, hidden, 0)
    dev = device if isinstance(device, torch.device) else torch.device(device)
    if dev.index is None:
        dev = torch.device(dev.type, torch.cuda.current_device())
    key = (dev, int(_raw_stream(dev, stream)))
    ws = _WORKSPACES.get(key)
    if ws is None or ws.numel() < need:
        s = stream if stream is not None else torch.cuda.current_stream(dev)
        with torch.cuda.stream(s):
            ws = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
        _WORKSPACES[key] = ws
    return ws


def forward(x, w_in, w_out, depth: int, n_trees: int = 1, y=None, *, y_dtype=None, **kw):
    """FFF forward through ``fff_forward_ex``; returns y (allocated if not given).

    In the modes that need scratch a cached workspace of the call's device and stream is passed
    unless ``workspace`` is given."""
    if y is None:
        y = torch.empty(x.shape, dtype=y_dtype or x.dtype, device=x.device)
    if kw.get("mode", "auto") in ("grouped", "auto", "tiled", "masked", 0, 2, 4, 5) and kw.get("workspace") is None:
        kw["workspace"] = workspace_for(x.shape[0], depth, n_trees, x.shape[1], x.device, kw.get("stream"))
    a = make_args(x, w_in, w_out, depth, n_trees, y, **kw)
    lib = load_library()
    with _on_device(x.device):
        _check(lib.fff_forward_ex(ctypes.byref(a)))
    return y


STATIC_SCRATCH_BYTES = 64 << 20  # FFF_STATIC_SCRATCH_BYTES


def forward_static(x, w_in, w_out, depth: int, n_trees: int = 1, y=None, *, y_dtype=None, **kw):
    """FFF forward through ``fff_forward_static``: the library's own scratch, nothing allocated by
    the call (y is allocated here if not given).  No ``workspace`` argument; MASKED unavailable."""
    if "workspace" in kw:
        raise ValueError("fff_forward_static takes no workspace")
    if y is None:
        y = torch.empty(x.shape, dtype=y_dtype or x.dtype, device=x.device)
    a = make_args(x, w_in, w_out, depth, n_trees, y, **kw)
    with torch.cuda.device(x.device):
        _check(load_library().fff_forward_static(ctypes.byref(a)))
    return y


def _stack_args(x, layers, depth, n_trees, y, kw):
    """fff_args and the fff_layer array of a stack; ``layers`` holds (W_in, W_out[, gamma[, beta]])."""
    if not layers:
        raise ValueError("a stack needs at least one layer")
    H = x.shape[1]
    arr = (FffLayer * len(layers))()
    w_dt = None
    for i, lay in enumerate(layers):
        w_in, w_out = lay[0], lay[1]
        gamma = lay[2] if len(lay) > 2 else None
        beta = lay[3] if len(lay) > 3 else None
        _check_weights(w_in, w_out, depth, n_trees, H, x.device)
        if w_dt is None:
            w_dt = w_in.dtype
        elif w_in.dtype != w_dt:
            raise ValueError("every layer's weights must share a dtype")
        arr[i].W_in, arr[i].W_out = w_in.data_ptr(), w_out.data_ptr()
        arr[i].norm_gamma = _check_norm_param(gamma, f"layer {i} gamma", H, x.device)
        arr[i].norm_beta = _check_norm_param(beta, f"layer {i} beta", H, x.device)
    kw.setdefault("out", "residual")
    a = make_args(x, None, None, depth, n_trees, y, n_layers=len(layers), **kw)
    a.w_dtype = _TORCH_DT[w_dt]
    return a, arr


def forward_stack(x, layers, depth: int, n_trees: int = 1, y=None, **kw):
    """Layers x <- x + FFF_i(norm_i(x)) through ``fff_forward_stack``; returns y (allocated if not given,
    of x's dtype; y may be x itself).  ``layers``: sequence of (W_in, W_out[, gamma[, beta]])."""
    if y is None:
        y = torch.empty_like(x)
    if kw.get("mode", "auto") in ("auto", "grouped", "tiled", "masked", 0, 2, 4, 5) and kw.get("workspace") is None:
        kw["workspace"] = workspace_for(x.shape[0], depth, n_trees, x.shape[1], x.device, kw.get("stream"))
    a, arr = _stack_args(x, layers, depth, n_trees, y, kw)
    with torch.cuda.device(x.device):
        _check(load_library().fff_forward_stack(ctypes.byref(a), arr, len(layers)))
    return y


def describe_stack(x, layers, depth: int, n_trees: int = 1, y=None, **kw) -> str:
    if y is None:
        y = torch.empty_like(x)
    if kw.get("mode", "auto") in ("auto", "grouped", "tiled", "masked", 0, 2, 4, 5) and kw.get("workspace") is None:
        kw["workspace"] = workspace_for(x.shape[0], depth, n_trees, x.shape[1], x.device, kw.get("stream"))
    a, arr = _stack_args(x, layers, depth, n_trees, y, kw)
    buf = ctypes.create_string_buffer(512)
    with torch.cuda.device(x.device):
        _check(load_library().fff_describe_stack(ctypes.byref(a), arr, len(layers), buf, len(buf)))
    return buf.value.decode()


_BWD_WORKSPACES: dict = {}


def backward_workspace_bytes(n_tokens: int, depth: int, n_trees: int, hidden: int) -> int:
    return int(load_library().fff_backward_workspace_bytes(n_tokens, depth, n_trees, hidden))


def backward(x, w_in, w_out, depth: int, n_trees: int, dy, leaves, logits, *, dx=None, dw_in=None, dw_out=None,
             act="gelu", accumulate=False, bad_leaves=None, workspace=None, stream=None, want=("dx", "dw_in", "dw_out"),
             dx_dtype=None):
    """Hard-routed backward through ``fff_backward``.

    ``leaves`` int32 [B, T] and ``logits`` float32 [B, T, D+1] come from the forward's records
    (``nodes_out[..., depth]`` and ``logits_out``).  Outputs named in ``want`` are allocated
    when not given (dx of ``dx_dtype`` or dy's dtype; dW in float32).  Returns (dx, dw_in, dw_out)."""
    device = dy.device
    B, H = dy.shape
    N = (1 << (depth + 1)) - 1
    _check_weights(w_in, w_out, depth, n_trees, H, device)
    _dev_tensor(dy, "dy", device)
    if x is not None:
        _dev_tensor(x, "x", device)
        if tuple(x.shape) != (B, H):
            raise ValueError("x and dy must have the same shape")
    for t, what, dt, n in ((leaves, "leaves", torch.int32, B * n_trees),
                           (logits, "logits", torch.float32, B * n_trees * (depth + 1))):
        _dev_tensor(t, what, device)
        if t.dtype != dt or t.numel() != n:
            raise ValueError(f"{what} must be {dt} with {n} elements")
    if dx is None and "dx" in want:
        dx = torch.empty((B, H), dtype=dx_dtype or dy.dtype, device=device)
    if dw_in is None and "dw_in" in want:
        dw_in = torch.empty((n_trees, N, H), dtype=torch.float32, device=device)
    if dw_out is None and "dw_out" in want:
        dw_out = torch.empty((n_trees, N, H), dtype=torch.float32, device=device)
    for t, what in ((dw_in, "dw_in"), (dw_out, "dw_out")):
        if t is not None:
            _dev_tensor(t, what, device)
            if t.dtype != torch.float32 or tuple(t.shape) != (n_trees, N, H):
                raise ValueError(f"{what} must be float32 [{n_trees}, {N}, {H}]")
    if dx is not None:
        _dev_tensor(dx, "dx", device)
    if (dw_in is not None or dw_out is not None) and workspace is None:
        need = backward_workspace_bytes(B, depth, n_trees, H)
        s = stream if stream is not None else torch.cuda.current_stream(device)
        key = (device, int(s.cuda_stream))  # one per (device, stream), as for the forward
        ws = _BWD_WORKSPACES.get(key)
        if ws is None or ws.numel() < need:
            with torch.cuda.stream(s):
                ws = torch.empty(max(need, 256), dtype=torch.uint8, device=device)
            _BWD_WORKSPACES[key] = ws
        workspace = ws
    a = FffBackwardArgs()
    a.x = x.data_ptr() if x is not None else None
    a.W_in, a.W_out, a.dy = w_in.data_ptr(), w_out.data_ptr(), dy.data_ptr()
    a.leaves, a.logits = leaves.data_ptr(), logits.data_ptr()
    a.dx = dx.data_ptr() if dx is not None else None
    a.dW_in = dw_in.data_ptr() if dw_in is not None else None
    a.dW_out = dw_out.data_ptr() if dw_out is not None else None
    a.n_tokens, a.hidden, a.depth, a.n_trees = B, H, depth, n_trees
    a.x_dtype = _dt(x, "x") if x is not None else FFF_F32
    a.w_dtype, a.dy_dtype = _dt(w_in, "W_in"), _dt(dy, "dy")
    a.dx_dtype = _dt(dx, "dx") if dx is not None else FFF_F32
    a.act = ACTS[act] if isinstance(act, str) else int(act)
    a.accumulate = int(bool(accumulate))
    if bad_leaves is not None:
        _dev_tensor(bad_leaves, "bad_leaves", device)
        a.bad_leaves = bad_leaves.data_ptr()
    if workspace is not None:
        a.workspace, a.workspace_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    a.hip_stream = (stream if stream is not None else torch.cuda.current_stream(device)).cuda_stream
    with torch.cuda.device(device):
        _check(load_library().fff_backward(ctypes.byref(a)))
    return dx, dw_in, dw_out


def forward_plain(x, w_in, w_out, depth: int, n_trees: int, y, stream=None):
    """The six-argument call ``fff_forward(x, W_in, W_out, depth, n_trees, y, ...)`` (exact GELU, store)."""
    a = make_args(x, w_in, w_out, depth, n_trees, y, stream=stream)
    lib = load_library()
    with torch.cuda.device(x.device):
        _check(lib.fff_forward(a.x, a.W_in, a.W_out, depth, n_trees, a.y, a.n_tokens, a.hidden, a.x_dtype,
                               a.w_dtype, a.y_dtype, a.hip_stream))
    return y


def describe(x, w_in, w_out, depth: int, n_trees: int = 1, y=None, **kw) -> str:
    """The kernel and launch shape ``forward`` would use."""
    if y is None:
        y = torch.empty(x.shape, dtype=kw.pop("y_dtype", None) or x.dtype, device=x.device)
    kw.pop("y_dtype", None)
    if kw.get("mode", "auto") in ("grouped", "auto", "tiled", "masked", 0, 2, 4, 5) and kw.get("workspace") is None:
        kw["workspace"] = workspace_for(x.shape[0], depth, n_trees, x.shape[1], x.device, kw.get("stream"))
    a = make_args(x, w_in, w_out, depth, n_trees, y, **kw)
    buf = ctypes.create_string_buffer(512)
    with torch.cuda.device(x.device):
        _check(load_library().fff_describe(ctypes.byref(a), buf, len(buf)))
    return buf.value.decode()


def workspace_bytes(n_tokens: int, depth: int, n_trees: int, hidden: int, split_level: int = 0) -> int:
    return int(load_library().fff_workspace_bytes(n_tokens, depth, n_trees, hidden, split_level))


def version() -> int:
    return int(load_library().fff_version())


def from_numpy(a, device) -> torch.Tensor:
    """numpy float32 / int32 array, or uint16 bf16 bit patterns, -> tensor on ``device``."""
    import numpy as np

    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def to_numpy(t: torch.Tensor):
    """Tensor -> numpy; bfloat16 comes back as uint16 bit patterns."""
    import numpy as np

    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()
