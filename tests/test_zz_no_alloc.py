"""fff_forward_static, the entry point that allocates nothing, through the C ABI.

Its output must equal fff_forward_ex's (same plan, same kernels; the scratch is
the library's static device array instead of the caller's workspace) bit for
bit, on two calls in a row, the second with a smaller input so that it runs on
the scratch the first left behind; both are also checked against the oracle on
sampled rows.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import parity
from paper_2311_10770_amd import synth
from tests.conftest import flush_print
from tests.gpu_util import DEV

pytestmark = pytest.mark.gpu


def _run_both(fff, L, depth, trees, y_dtype, mode):
    x, wi, wo = (fff.from_numpy(L[k], DEV) for k in ("x", "w_in", "w_out"))
    B, H = L["x"].shape
    ydt = torch.bfloat16 if y_dtype == "bf16" else torch.float32
    out = {}
    for name, fn in (("ex", fff.forward), ("static", fff.forward_static)):
        y = torch.full((B, H), float("nan"), dtype=ydt, device=DEV)
        nodes = torch.full((B, trees, depth + 1), -7, dtype=torch.int32, device=DEV)
        fn(x, wi, wo, depth, trees, y, nodes_out=nodes, mode=mode)
        torch.cuda.synchronize()
        out[name] = (fff.to_numpy(y), nodes.cpu().numpy())
    return out


def _check_sample(L, depth, trees, y_np, nodes_np, tol, n=1536):
    B = L["x"].shape[0]
    rows = np.sort(np.random.default_rng(B).choice(B, min(n, B), replace=False))
    ref = oracle.forward(L["x"][rows], L["w_in"], L["w_out"], depth, trees)
    return parity.assert_parity(L["x"], L["w_in"], L["w_out"], depth, trees, ref, y_np, nodes_np, tol=tol,
                                rows=rows)


@pytest.mark.parametrize("mode", ["tiled", "auto"])
def test_static_equals_ex_on_two_calls(fff_lib, mode):
    """Headline shape (depth 11, hidden 768, bf16) at 65536 tokens, then 20000 clustered tokens
    whose crowded leaves overflow their buckets, in that order."""
    w_in, w_out = synth.make_weights(3, 768, 11, 1, "bf16")
    first = {"x": synth.make_x(3, 65536, 768, "bf16"), "w_in": w_in, "w_out": w_out}
    second = {"x": synth.make_clustered_x(7, 20000, 768, "bf16", n_centres=8), "w_in": w_in, "w_out": w_out}
    for label, L in (("65536 tokens", first), ("20000 clustered tokens", second)):
        flush_print(f"[gpu] static vs ex, mode={mode}, {label}")
        got = _run_both(fff_lib, L, 11, 1, "bf16", mode)
        assert np.array_equal(got["ex"][0], got["static"][0]), label
        assert np.array_equal(got["ex"][1], got["static"][1]), label
        rep = _check_sample(L, 11, 1, got["static"][0], got["static"][1], 2e-2)
        flush_print(f"[gpu] static {label}: {parity.summary(rep)}")


def test_static_grouped_fp32_two_calls(fff_lib):
    """The grouped plan (fp32, 16384 tokens, then 3000) on the static scratch."""
    w_in, w_out = synth.make_weights(2, 768, 11, 1, "f32")
    for B in (16384, 3000):
        L = {"x": synth.make_x(2, B, 768, "f32"), "w_in": w_in, "w_out": w_out}
        flush_print(f"[gpu] static grouped fp32 B={B}")
        got = _run_both(fff_lib, L, 11, 1, "f32", "grouped")
        assert np.array_equal(got["ex"][0], got["static"][0]) and np.array_equal(got["ex"][1], got["static"][1])
        _check_sample(L, 11, 1, got["static"][0], got["static"][1], 1e-5)


def test_static_limits(fff_lib):
    """No workspace argument, no MASKED, and an explicit plan whose scratch exceeds the array is
    refused before anything runs; AUTO then takes a plan that fits."""
    fff = fff_lib
    L = synth.make_layer(9, 512, 768, 3, 16, "bf16", "bf16")
    x, wi, wo = (fff.from_numpy(L[k], DEV) for k in ("x", "w_in", "w_out"))
    with pytest.raises(fff.FffError) as e:
        fff.forward_static(x, wi, wo, 3, 16, mode="masked")
    assert e.value.status == fff.fff.FFF_ERR_UNSUPPORTED
    y_auto = fff.forward_static(x, wi, wo, 3, 16)  # AUTO would pick masked in fff_forward_ex
    y_ref = fff.forward(x, wi, wo, 3, 16, mode="descent")
    torch.cuda.synchronize()
    assert torch.equal(y_auto, y_ref)
    a = fff.make_args(x, wi, wo, 3, 16, torch.empty_like(x))
    ws = torch.empty(1 << 20, dtype=torch.uint8, device=DEV)
    a.workspace, a.workspace_bytes = ws.data_ptr(), ws.numel()
    assert fff.load_library().fff_forward_static(a) == fff.fff.FFF_ERR_INVALID_ARG
    B = 262144  # the tiled scratch of 262144 tokens at depth 11 is 82 MiB
    assert fff.workspace_bytes(B, 11, 1, 768) > fff.fff.STATIC_SCRATCH_BYTES
    xb = torch.zeros((B, 768), dtype=torch.bfloat16, device=DEV)
    w11 = fff.from_numpy(synth.make_weights(3, 768, 11, 1, "bf16")[0], DEV)
    with pytest.raises(fff.FffError) as e:
        fff.forward_static(xb, w11, w11, 11, 1, mode="tiled")
    assert e.value.status == fff.fff.FFF_ERR_WORKSPACE
