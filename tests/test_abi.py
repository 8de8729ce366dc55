"""The C ABI without a GPU: exports, struct layout, and argument validation.

Every call here fails validation (or is a zero-token no-op), which the ABI
promises happens before any HIP call, so nothing touches a device.
"""
import ctypes
import re
import subprocess

import pytest

from paper_2311_10770_amd import build as native_build
from paper_2311_10770_amd import fff as binding
from tests.conftest import ROOT

HEADER = ROOT / "include" / "fff.h"


def declared_functions():
    text = re.sub(r"/\*.*?\*/", "", HEADER.read_text(), flags=re.S)
    return sorted(set(re.findall(r"\b(fff_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not binding.LIB_PATH.exists():
        native_build.build_lib("libfff.so")
    return binding.load_library()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert set(names) == set(binding.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", str(binding.LIB_PATH)], capture_output=True, text=True,
                         check=True).stdout
    exported = {ln.split()[-1] for ln in out.splitlines() if " T " in ln}
    assert set(names) <= exported
    assert not {e for e in exported if not e.startswith("fff_") and not e.startswith("_init")
                and not e.startswith("_fini")}, "only the fff_ ABI is exported"


@pytest.mark.parametrize("cls,cname", [(binding.FffArgs, "fff_args"), (binding.FffLayer, "fff_layer"),
                                       (binding.FffBackwardArgs, "fff_backward_args")])
def test_struct_layout_matches_c(tmp_path, cls, cname):
    fields = [f[0] for f in cls._fields_]
    src = tmp_path / "layout.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "fff.h"\nint main(void){\n'
                   + f'printf("%zu\\n", sizeof({cname}));\n'
                   + "".join(f'printf("%zu\\n", offsetof({cname}, {f}));\n' for f in fields) + "return 0;}\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", str(ROOT / "include"), str(src), "-o", str(exe)], check=True)
    vals = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split()]
    assert vals[0] == ctypes.sizeof(cls)
    assert len(vals) - 1 == len(fields)
    for f, off in zip(fields, vals[1:]):
        assert getattr(cls, f).offset == off, f


def test_version_and_status_strings(lib):
    assert lib.fff_version() == 101
    for rc in (0, -1, -2, -3, -4):
        assert lib.fff_status_str(rc).decode().startswith("FFF_")
    assert lib.fff_status_str(7) == b"unknown fff status"
    assert lib.fff_last_hip_error() == 0


P = 0x100000  # an aligned fake device address; validation never dereferences it


def good_args(**over):
    a = binding.FffArgs()
    a.x, a.W_in, a.W_out, a.y = P, P * 16, P * 16, P * 64
    a.n_tokens, a.hidden, a.depth, a.n_trees = 4, 64, 3, 1
    for k, v in over.items():
        setattr(a, k, v)
    return a


@pytest.mark.parametrize("over", [
    dict(n_tokens=-1), dict(hidden=0), dict(depth=-1), dict(depth=25), dict(n_trees=0),
    dict(x_dtype=2), dict(w_dtype=-1), dict(y_dtype=5), dict(act=3), dict(mode=9), dict(mode=7), dict(mode=-1), dict(out_mode=3),
    dict(lds_levels=-2), dict(split_level=4), dict(split_level=-2),
    dict(x=None), dict(W_in=None), dict(W_out=None), dict(y=None),
    dict(x=P + 4), dict(y=P * 64 + 8), dict(W_in=P * 16 + 2),
    dict(y=P + 64),                           # overlaps x
    dict(nodes_out=P * 64 + 16),              # overlaps y
    dict(nodes_out=P * 256, logits_out=P * 256 + 16),
    dict(n_tokens=1 << 62),                   # size overflow
    dict(y=P * 16 + 64),                      # output overlaps the weights
    dict(nodes_out=P + 32),                   # records overlap x
    dict(y=P, y_dtype=1),                     # in place needs one dtype
    dict(norm=2), dict(norm=1, norm_eps=-1.0), dict(norm=1, norm_eps=float("nan")),
    dict(norm=1, norm_eps=float("inf")),
    dict(norm=1, norm_gamma=P * 128 + 4),     # misaligned gain
    dict(norm=1, norm_beta=P * 64 + 256),     # shift overlaps y
])
def test_invalid_arguments_rejected_before_hip(lib, over):
    a = good_args(**over)
    assert lib.fff_forward_ex(ctypes.byref(a)) == binding.FFF_ERR_INVALID_ARG
    buf = ctypes.create_string_buffer(64)
    assert lib.fff_describe(ctypes.byref(a), buf, len(buf)) == binding.FFF_ERR_INVALID_ARG
    assert lib.fff_last_hip_error() == 0


def test_null_args_and_zero_tokens(lib):
    assert lib.fff_forward_ex(None) == binding.FFF_ERR_INVALID_ARG
    a = binding.FffArgs()
    a.n_tokens, a.hidden, a.depth, a.n_trees = 0, 768, 11, 1
    assert lib.fff_forward_ex(ctypes.byref(a)) == binding.FFF_OK  # no pointers needed, nothing enqueued
    assert lib.fff_forward(None, None, None, 11, 1, None, 0, 768, 0, 0, 0, None) == binding.FFF_OK
    assert lib.fff_forward(None, None, None, 11, 1, None, 5, 768, 0, 0, 0, None) == binding.FFF_ERR_INVALID_ARG


def test_workspace_bytes_rejects_bad_shapes(lib):
    assert lib.fff_workspace_bytes(-1, 11, 1, 768, 0) == 0
    assert lib.fff_workspace_bytes(100, 25, 1, 768, 0) == 0
    assert lib.fff_workspace_bytes(100, 11, 0, 768, 0) == 0
    assert lib.fff_workspace_bytes(100, 11, 1, 768, 12) == 0


def test_build_flags_disable_packed_fp32():
    flags = " ".join(native_build.COMMON)
    assert "-packed-fp32-ops" in flags and "--offload-arch=gfx950" in flags


def stack_args(**over):
    a = good_args(out_mode=binding.OUTS["residual"])
    a.W_in = a.W_out = None
    for k, v in over.items():
        setattr(a, k, v)
    return a


def layers(n, **over):
    arr = (binding.FffLayer * max(n, 1))()
    for i in range(n):
        arr[i].W_in, arr[i].W_out = P * (16 + 8 * i), P * (20 + 8 * i)
        for k, v in over.items():
            setattr(arr[i], k, v)
    return arr


@pytest.mark.parametrize("over,lover,n", [
    ({}, {}, 0),                                            # no layers
    (dict(W_in=P * 16), {}, 2),                             # weights come from the layer table
    (dict(norm_gamma=P * 128), {}, 2),
    (dict(out_mode=0), {}, 2),                              # a stack is residual
    (dict(y_dtype=1), {}, 2),                               # one residual-stream dtype
    ({}, dict(W_out=None), 2),
    ({}, dict(W_in=P * 16 + 8), 2),
    (dict(norm=1), dict(norm_gamma=P * 128 + 4), 2),
    ({}, dict(W_in=P * 64), 2),                             # weights overlap y
    (dict(nodes_out=P * 256, logits_out=P * 256 + 4 * 4 * 4 * 2), {}, 3),  # records of 3 layers overlap
])
def test_stack_invalid_arguments(lib, over, lover, n):
    a = stack_args(**over)
    arr = layers(n, **lover)
    assert lib.fff_forward_stack(ctypes.byref(a), arr, n) == binding.FFF_ERR_INVALID_ARG
    buf = ctypes.create_string_buffer(64)
    assert lib.fff_describe_stack(ctypes.byref(a), arr, n, buf, len(buf)) == binding.FFF_ERR_INVALID_ARG
    assert lib.fff_last_hip_error() == 0


def test_stack_null_table_and_zero_tokens(lib):
    a = stack_args()
    assert lib.fff_forward_stack(ctypes.byref(a), None, 2) == binding.FFF_ERR_INVALID_ARG
    assert lib.fff_forward_stack(None, layers(1), 1) == binding.FFF_ERR_INVALID_ARG
    a.n_tokens = 0
    assert lib.fff_forward_stack(ctypes.byref(a), layers(3), 3) == binding.FFF_OK


def bwd_args(**over):
    a = binding.FffBackwardArgs()
    a.x, a.W_in, a.W_out, a.dy = P, P * 16, P * 24, P * 32
    a.leaves, a.logits = P * 40, P * 48
    a.dx, a.dW_in, a.dW_out = P * 64, P * 80, P * 96
    a.n_tokens, a.hidden, a.depth, a.n_trees = 4, 64, 3, 1
    a.workspace, a.workspace_bytes = P * 256, 1 << 20
    for k, v in over.items():
        setattr(a, k, v)
    return a


@pytest.mark.parametrize("over", [
    dict(hidden=66), dict(hidden=0), dict(depth=25), dict(n_trees=0), dict(n_tokens=-1), dict(dy_dtype=2),
    dict(dx_dtype=-1), dict(act=5), dict(accumulate=2),
    dict(W_out=None), dict(dy=None), dict(leaves=None), dict(logits=None), dict(x=None),  # x needed for dW_in
    dict(dx=P * 64 + 8), dict(leaves=P * 40 + 2),
    dict(dx=P * 32 + 64),                      # dx overlaps dy
    dict(dW_in=P * 96),                        # dW_in is dW_out
    dict(dW_out=P * 16),                       # dW_out overwrites W_in
    dict(workspace=P * 64),                    # workspace overlaps dx
    dict(n_tokens=1 << 40),                    # tokens x trees past int32
])
def test_backward_invalid_arguments(lib, over):
    a = bwd_args(**over)
    assert lib.fff_backward(ctypes.byref(a)) == binding.FFF_ERR_INVALID_ARG
    assert lib.fff_last_hip_error() == 0


def test_backward_workspace_rules(lib):
    need = lib.fff_backward_workspace_bytes(4, 3, 1, 64)
    assert need > 0 and lib.fff_backward_workspace_bytes(-1, 3, 1, 64) == 0
    assert lib.fff_backward_workspace_bytes(4, 25, 1, 64) == 0 and lib.fff_backward_workspace_bytes(4, 3, 1, 0) == 0
    for over in (dict(workspace=None), dict(workspace_bytes=need - 1), dict(workspace=P * 256 + 16)):
        assert lib.fff_backward(ctypes.byref(bwd_args(**over))) == binding.FFF_ERR_WORKSPACE
    # dx only needs no workspace, and nothing requested or no tokens is a no-op
    a = bwd_args(dW_in=None, dW_out=None, workspace=None, workspace_bytes=0, n_tokens=0)
    assert lib.fff_backward(ctypes.byref(a)) == binding.FFF_OK
    a = bwd_args(dx=None, dW_in=None, dW_out=None)
    assert lib.fff_backward(ctypes.byref(a)) == binding.FFF_OK
    assert lib.fff_backward(None) == binding.FFF_ERR_INVALID_ARG


def test_binding_modes_match_header():
    """The binding's mode names carry the header's fff_mode values, one for one."""
    text = HEADER.read_text()
    enum = {m.lower(): int(v) for m, v in re.findall(r"FFF_MODE_([A-Z]+)\s*=\s*(\d+)", text)}
    assert enum == binding.MODES
