"""GPU parity of the layer context: LayerNorm prologue, residual epilogue,
in-place calls and stacks of layers (x <- x + FFF_i(LN_i(x))).

* single layers against the oracle's block (LayerNorm in fp64, then the FFF,
  then the residual), in every mode and type combination;
* in-place calls (y is x) against out-of-place ones, bit for bit;
* the persistent stack kernel against chained single-layer calls, bit for
  bit (same arithmetic per layer), and the chained calls against the oracle
  layer by layer on the device's own intermediate values (teacher forcing);
* the 12-layer stack of UltraFastBERT-4x9 layers at 16384 tokens.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import parity
from paper_2311_10770_amd import synth
from paper_2311_10770_amd.configs import WORKLOADS
from tests.conftest import flush_print
from tests.gpu_util import DEV, TORCH_DT

pytestmark = pytest.mark.gpu

EPS = 1e-5


def dev(fff, a):
    return fff.from_numpy(a, DEV)


def check_block(fff, name, x, wi, wo, depth, trees, y_dtype, *, norm, out, mode, gamma=None, beta=None,
                eps=EPS, in_place=False):
    """One layer on the device vs the oracle's block; returns the device output (numpy)."""
    B, H = x.shape
    flush_print(f"[gpu] {name}: B={B} H={H} depth={depth} trees={trees} y={y_dtype} norm={norm} out={out} "
                f"mode={mode} in_place={in_place}")
    xd = dev(fff, x)
    y = xd if in_place else torch.full((B, H), float("nan"), dtype=TORCH_DT[y_dtype], device=DEV)
    nodes = torch.full((B, trees, depth + 1), -7, dtype=torch.int32, device=DEV)
    kw = {}
    if norm:
        kw = dict(norm="layernorm", norm_eps=eps, norm_gamma=None if gamma is None else dev(fff, gamma),
                  norm_beta=None if beta is None else dev(fff, beta))
    fff.forward(xd, dev(fff, wi), dev(fff, wo), depth, trees, y, out=out, mode=mode, nodes_out=nodes, **kw)
    torch.cuda.synchronize()
    got = fff.to_numpy(y)
    ref = oracle.block(x, wi, wo, depth, trees, norm={"gamma": gamma, "beta": beta, "eps": eps} if norm else None)
    u = ref["u"]
    nd = nodes.cpu().numpy()
    residual = out == "residual"
    # a bf16 output that stores x + FFF(u) is judged on the stored total: normwise 2e-2 and, per
    # element, one bf16 spacing of the fp64 total plus the fp32 bar on FFF(u)
    tol = 2e-2 if y_dtype == "bf16" else 1e-5
    fff_only = {k: ref[k] for k in ("nodes", "logits", "near_tie")}
    fff_only["y"] = ref["fff"]
    rep = parity.assert_parity(u, wi, wo, depth, trees, fff_only, got, nd, tol=tol,
                               base_dev=x if residual else None)
    flush_print(f"[gpu] {name}: ok, {parity.summary(rep)}")
    return got


NORM_COMBOS = [("f32", "f32", "f32"), ("bf16", "bf16", "bf16"), ("f32", "bf16", "f32"), ("bf16", "f32", "bf16"),
               ("bf16", "bf16", "f32")]


@pytest.mark.parametrize("xd,wd,yd", NORM_COMBOS)
@pytest.mark.parametrize("mode", ["descent", "grouped", "generic"])
@pytest.mark.parametrize("out", ["residual", "store"])
def test_layernorm_layer(fff_lib, xd, wd, yd, mode, out):
    B, H, D, T = 1000, 768, 9, 1
    L = synth.make_layer(200, B, H, D, T, xd, wd)
    gamma, beta = synth.make_norm(200, H)
    check_block(fff_lib, f"LN {xd}/{wd}/{yd}", L["x"], L["w_in"], L["w_out"], D, T, yd, norm=True, out=out,
                mode=mode, gamma=gamma, beta=beta)


@pytest.mark.parametrize("H", [1024, 4096, 100])
@pytest.mark.parametrize("wd", ["f32", "bf16"])
def test_layernorm_other_widths(fff_lib, H, wd):
    D = 6 if H == 4096 else 8
    L = synth.make_layer(210 + H, 300, H, D, 2, wd, wd)
    gamma, beta = synth.make_norm(210 + H, H)
    check_block(fff_lib, f"LN H={H} {wd}", L["x"], L["w_in"], L["w_out"], D, 2, wd, norm=True, out="residual",
                mode="auto", gamma=gamma, beta=beta)


def test_layernorm_without_affine_and_bert_eps(fff_lib):
    L = synth.make_layer(220, 777, 768, 11, 1, "f32", "bf16")
    check_block(fff_lib, "LN no affine", L["x"], L["w_in"], L["w_out"], 11, 1, "f32", norm=True, out="residual",
                mode="auto", eps=1e-12)


def test_layernorm_scale_invariance_on_device(fff_lib):
    """LN makes the layer blind to a positive scale and a shift of x (eps = 0): same paths, same FFF part."""
    x = synth.make_x(230, 512, 768, "f32")
    wi, wo = synth.make_weights(230, 768, 10, 1, "f32")
    kw = dict(norm="layernorm", norm_eps=0.0, mode="descent")
    n1 = torch.empty((512, 1, 11), dtype=torch.int32, device=DEV)
    n2 = torch.empty_like(n1)
    y1 = fff_lib.forward(dev(fff_lib, x), dev(fff_lib, wi), dev(fff_lib, wo), 10, 1, nodes_out=n1, **kw)
    x2 = (x * np.float32(4.0) + np.float32(0.5)).astype(np.float32)
    y2 = fff_lib.forward(dev(fff_lib, x2), dev(fff_lib, wi), dev(fff_lib, wo), 10, 1, nodes_out=n2, **kw)
    torch.cuda.synchronize()
    same = (n1 == n2).all(dim=(1, 2))
    assert same.float().mean() > 0.99  # rounding of the rescaled input may flip a rare near tie
    err = (y1[same] - y2[same]).norm(dim=1) / y1[same].norm(dim=1)
    assert float(err.max()) < 1e-5


@pytest.mark.parametrize("mode", ["descent", "grouped", "generic"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("norm", [False, True])
def test_in_place_equals_out_of_place(fff_lib, mode, dt, norm):
    L = synth.make_layer(240, 3001, 768, 11, 1, dt, dt)
    gamma, beta = synth.make_norm(240, 768)
    wi, wo = dev(fff_lib, L["w_in"]), dev(fff_lib, L["w_out"])
    kw = dict(mode=mode, out="residual")
    if norm:
        kw.update(norm="layernorm", norm_eps=EPS, norm_gamma=dev(fff_lib, gamma), norm_beta=dev(fff_lib, beta))
    x = dev(fff_lib, L["x"])
    y = fff_lib.forward(x, wi, wo, 11, 1, torch.empty_like(x), **kw)
    z = x.clone()
    fff_lib.forward(z, wi, wo, 11, 1, z, **kw)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16) if dt == "bf16" else y, z.view(torch.int16) if dt == "bf16" else z)


# ----------------------------------------------------------------------- stacks


def make_stack(seed, n_layers, H, D, T, wd, norm):
    layers = []
    for i in range(n_layers):
        wi, wo = synth.make_weights(seed, H, D, T, wd, layer=i + 1)
        g, b = synth.make_norm(seed, H, layer=i + 1) if norm else (None, None)
        layers.append({"w_in": wi, "w_out": wo, "gamma": g, "beta": b})
    return layers


def dev_layers(fff, layers, norm):
    out = []
    for lay in layers:
        t = [dev(fff, lay["w_in"]), dev(fff, lay["w_out"])]
        if norm:
            t += [dev(fff, lay["gamma"]), dev(fff, lay["beta"])]
        out.append(tuple(t))
    return out


def chained(fff, x, dlayers, D, T, norm, mode, records=False):
    """The stack as single-layer calls, in place on y after the first layer."""
    B = x.shape[0]
    y = torch.empty_like(x)
    outs, nodes = [], []
    cur = x
    for lay in dlayers:
        kw = dict(mode=mode, out="residual")
        if norm:
            kw.update(norm="layernorm", norm_eps=EPS, norm_gamma=lay[2], norm_beta=lay[3])
        nd = torch.empty((B, T, D + 1), dtype=torch.int32, device=DEV) if records else None
        fff.forward(cur, lay[0], lay[1], D, T, y, nodes_out=nd, **kw)
        if records:
            outs.append(y.clone())
            nodes.append(nd)
        cur = y
    return y, outs, nodes


def bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t


STACK_COMBOS = [("f32", "f32"), ("bf16", "bf16"), ("f32", "bf16"), ("bf16", "f32")]


@pytest.mark.parametrize("xd,wd", STACK_COMBOS)
@pytest.mark.parametrize("norm", [False, True])
def test_stack_kernel_equals_chained_calls(fff_lib, xd, wd, norm):
    B, H, D, T, NL = 2053, 768, 9, 2, 4
    x = dev(fff_lib, synth.make_x(250, B, H, xd))
    dl = dev_layers(fff_lib, make_stack(250, NL, H, D, T, wd, norm), norm)
    kw = dict(norm="layernorm", norm_eps=EPS) if norm else {}
    flush_print(f"[gpu] stack {xd}/{wd} norm={norm}: {fff_lib.describe_stack(x, dl, D, T, mode='descent', **kw)}")
    nodes = torch.empty((NL, B, T, D + 1), dtype=torch.int32, device=DEV)
    ys = fff_lib.forward_stack(x, dl, D, T, mode="descent", nodes_out=nodes, **kw)
    yc, _, nc = chained(fff_lib, x, dl, D, T, norm, "descent", records=True)
    torch.cuda.synchronize()
    assert torch.equal(bits(ys), bits(yc))
    assert torch.equal(nodes, torch.stack(nc))


@pytest.mark.parametrize("mode", ["grouped", "generic"])
def test_stack_per_layer_modes_equal_chained_calls(fff_lib, mode):
    B, H, D, T, NL = 999, 768, 11, 1, 3
    x = dev(fff_lib, synth.make_x(255, B, H, "bf16"))
    dl = dev_layers(fff_lib, make_stack(255, NL, H, D, T, "bf16", True), True)
    kw = dict(norm="layernorm", norm_eps=EPS)
    assert fff_lib.describe_stack(x, dl, D, T, mode=mode, **kw).startswith("per-layer")
    ys = fff_lib.forward_stack(x, dl, D, T, mode=mode, **kw)
    yc, _, _ = chained(fff_lib, x, dl, D, T, True, mode)
    torch.cuda.synchronize()
    assert torch.equal(bits(ys), bits(yc))


@pytest.mark.parametrize("B", [1, 5, 64, 1000])
@pytest.mark.parametrize("NL", [1, 2, 35])
def test_stack_ragged_and_long(fff_lib, B, NL):
    """Token counts that leave idle waves and workgroups; more layers than one launch carries."""
    H, D, T = 768, 5, 1
    x = dev(fff_lib, synth.make_x(260, B, H, "f32"))
    dl = dev_layers(fff_lib, make_stack(260, NL, H, D, T, "bf16", True), True)
    kw = dict(norm="layernorm", norm_eps=EPS)
    ys = fff_lib.forward_stack(x, dl, D, T, mode="descent", **kw)
    yc, _, _ = chained(fff_lib, x, dl, D, T, True, "descent")
    z = x.clone()
    fff_lib.forward_stack(z, dl, D, T, z, mode="descent", **kw)  # in place
    torch.cuda.synchronize()
    assert torch.equal(ys, yc) and torch.equal(ys, z)


@pytest.mark.parametrize("xd,wd", [("f32", "f32"), ("bf16", "bf16")])
def test_stack_layers_teacher_forced_against_oracle(fff_lib, xd, wd):
    """Each chained layer (bitwise the stack kernel's) against the oracle block on its own device input."""
    B, H, D, T, NL = 1500, 768, 9, 4, 3
    xs = synth.make_x(270, B, H, xd)
    layers = make_stack(270, NL, H, D, T, wd, True)
    dl = dev_layers(fff_lib, layers, True)
    _, outs, nodes = chained(fff_lib, dev(fff_lib, xs), dl, D, T, True, "descent", records=True)
    torch.cuda.synchronize()
    cur = xs
    for i, lay in enumerate(layers):
        got = fff_lib.to_numpy(outs[i])
        nd = nodes[i].cpu().numpy()
        ref = oracle.block(cur, lay["w_in"], lay["w_out"], D, T,
                           norm={"gamma": lay["gamma"], "beta": lay["beta"], "eps": EPS})
        fff_only = {k: ref[k] for k in ("nodes", "logits", "near_tie")}
        fff_only["y"] = ref["fff"]
        rep = parity.assert_parity(ref["u"], lay["w_in"], lay["w_out"], D, T, fff_only, got, nd,
                                   tol=2e-2 if xd == "bf16" else 1e-5, base_dev=cur)
        flush_print(f"[gpu] layer {i}: ok, {parity.summary(rep)}")
        cur = got


def test_twelve_layer_4x9_stack_full_size(fff_lib):
    """The 12 stacked UltraFastBERT-4x9 layers at 16384 tokens (fp32), with LayerNorm: stack kernel ==
    chained calls, and the last layer against the oracle on its device input."""
    w = WORKLOADS["4x9_h768_b16384_f32_x12"]
    B, H, D, T, NL = w.n_tokens, w.hidden, w.depth, w.n_trees, w.layers
    xs = synth.make_x(w.seed, B, H, "f32")
    layers = make_stack(w.seed, NL, H, D, T, "f32", True)
    dl = dev_layers(fff_lib, layers, True)
    x = dev(fff_lib, xs)
    kw = dict(norm="layernorm", norm_eps=EPS)
    flush_print(f"[gpu] 12x 4x9: {fff_lib.describe_stack(x, dl, D, T, mode='descent', **kw)}")
    # AUTO: per-layer launches, leaf-tiled (four fp32 trees of depth 9, 32 tokens per leaf)
    assert fff_lib.describe_stack(x, dl, D, T, **kw).startswith("per-layer tiled")
    ys = fff_lib.forward_stack(x, dl, D, T, mode="descent", **kw)
    yc, outs, nodes = chained(fff_lib, x, dl, D, T, True, "descent", records=True)
    ya, _, _ = chained(fff_lib, x, dl, D, T, True, "auto")
    torch.cuda.synchronize()
    assert torch.equal(ys, yc)
    assert torch.equal(fff_lib.forward_stack(x, dl, D, T, **kw), ya)
    rows = np.random.default_rng(0).choice(B, 1024, replace=False)
    x_last = fff_lib.to_numpy(outs[-2])[rows]
    lay = layers[-1]
    ref = oracle.block(x_last, lay["w_in"], lay["w_out"], D, T,
                       norm={"gamma": lay["gamma"], "beta": lay["beta"], "eps": EPS})
    fff_only = {k: ref[k] for k in ("nodes", "logits", "near_tie")}
    fff_only["y"] = ref["fff"]
    parity.assert_parity(ref["u"], lay["w_in"], lay["w_out"], D, T, fff_only, fff_lib.to_numpy(ys)[rows],
                         nodes[-1].cpu().numpy()[rows], tol=1e-5, base_dev=x_last)
