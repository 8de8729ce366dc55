"""GPU parity of the hard-routed backward (fff_backward) against the fp64 oracle.

* exact: identity activation on small integers, where every product and sum
  is an integer that fp32 holds exactly -- dx, dW_in and dW_out must match the
  oracle bit for bit, whatever the summation order (this pins that every
  (token, level) term lands in the right row exactly once, root row included);
* bounded: GELU on Gaussian inputs, against first-order fp32 rounding bounds
  that hold for any summation order (``oracle.parity.backward_check``);
* the forward's own records as inputs (device path), out-of-range leaves,
  accumulation, every type combination, generic widths, and the 65536-token
  depth-11 layer.
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


def dev(fff, a):
    return fff.from_numpy(np.ascontiguousarray(a), DEV)


def run_bwd(fff, L, D, T, dy, leaves, logits32, *, act="gelu", dx_dtype="f32", accumulate=False, init=None,
            bad=None):
    B, H = L["x"].shape
    kw = {}
    if init is not None:
        kw = dict(dx=dev(fff, init["dx"]), dw_in=dev(fff, init["dw_in"]), dw_out=dev(fff, init["dw_out"]))
    dx, dwi, dwo = fff.backward(dev(fff, L["x"]), dev(fff, L["w_in"]), dev(fff, L["w_out"]), D, T, dev(fff, dy),
                                dev(fff, leaves), dev(fff, logits32), act=act, accumulate=accumulate,
                                dx_dtype=torch.bfloat16 if dx_dtype == "bf16" else torch.float32,
                                bad_leaves=bad, **kw)
    torch.cuda.synchronize()
    return {"dx": fff.to_numpy(dx), "dw_in": fff.to_numpy(dwi), "dw_out": fff.to_numpy(dwo)}


def int_layer(seed, B, H, D, T, dtype):
    rng = np.random.default_rng(seed)
    N = (1 << (D + 1)) - 1
    cast = (lambda a: synth.as_dtype(a.astype(np.float32), dtype))
    return {"x": cast(rng.integers(-3, 4, (B, H))), "w_in": cast(rng.integers(-3, 4, (T, N, H))),
            "w_out": cast(rng.integers(-3, 4, (T, N, H)))}


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("B,H,D,T", [(4096, 64, 11, 1), (300, 768, 9, 4), (77, 1024, 5, 2), (50, 100, 4, 3),
                                     (1000, 768, 0, 16)])
def test_exact_small_integers(fff_lib, dtype, B, H, D, T):
    L = int_layer(B + H + D, B, H, D, T, dtype)
    dy = synth.as_dtype(np.random.default_rng(1).integers(-3, 4, (B, H)).astype(np.float32), dtype)
    fwd = oracle.forward(L["x"], L["w_in"], L["w_out"], D, T, act="identity")
    leaves = fwd["nodes"][:, :, D].astype(np.int32)
    flush_print(f"[gpu] exact bwd {dtype} B={B} H={H} D={D} T={T}")
    got = run_bwd(fff_lib, L, D, T, dy, leaves, fwd["logits"].astype(np.float32), act="identity")
    ref = oracle.backward(L["x"], L["w_in"], L["w_out"], D, T, dy, fwd["nodes"], act="identity")
    for k in ("dx", "dw_in", "dw_out"):
        assert np.array_equal(got[k].astype(np.float64), ref[k]), k


def bounded_case(fff, name, L, D, T, dy, act="gelu", dx_dtype="f32", path_from="oracle"):
    B, H = L["x"].shape
    flush_print(f"[gpu] bwd {name}: B={B} H={H} D={D} T={T} act={act} dx={dx_dtype} path={path_from}")
    if path_from == "oracle":
        fwd = oracle.forward(L["x"], L["w_in"], L["w_out"], D, T, act=act)
        nodes, logits32 = fwd["nodes"], fwd["logits"].astype(np.float32)
    else:  # the device forward's own records
        x, wi, wo = dev(fff, L["x"]), dev(fff, L["w_in"]), dev(fff, L["w_out"])
        nd = torch.empty((B, T, D + 1), dtype=torch.int32, device=DEV)
        lg = torch.empty((B, T, D + 1), dtype=torch.float32, device=DEV)
        fff.forward(x, wi, wo, D, T, act=act, nodes_out=nd, logits_out=lg, y_dtype=torch.float32)
        torch.cuda.synchronize()
        nodes, logits32 = nd.cpu().numpy(), lg.cpu().numpy()
    got = run_bwd(fff, L, D, T, dy, nodes[:, :, D].copy(), logits32, act=act, dx_dtype=dx_dtype)
    ref = oracle.backward(L["x"], L["w_in"], L["w_out"], D, T, dy, nodes, act=act)
    rep = parity.backward_check(L["x"], L["w_in"], L["w_out"], D, T, dy, nodes, logits32, got, ref, act=act)
    assert rep["ok"], rep["fail"]
    flush_print(f"[gpu] bwd {name}: ok, dW_out err/scale {rep['dw_out_max_err_over_scale']:.2e} "
                f"(err/bound {rep['dw_out_max_err_over_bound']:.2f}), dW_in err/scale "
                f"{rep['dw_in_max_err_over_scale']:.2e} (err/bound {rep['dw_in_max_err_over_bound']:.2f}), "
                f"dx err/norm {rep['dx_max_err_over_norm']:.2e}")
    return rep


COMBOS = [("f32", "f32", "f32", "f32"), ("bf16", "bf16", "bf16", "f32"), ("bf16", "bf16", "bf16", "bf16"),
          ("f32", "bf16", "f32", "f32"), ("bf16", "f32", "f32", "bf16")]


@pytest.mark.parametrize("xd,wd,dyd,dxd", COMBOS)
@pytest.mark.parametrize("H", [768, 1024, 4096])
def test_bounded_type_combinations(fff_lib, xd, wd, dyd, dxd, H):
    D = 6 if H == 4096 else 9
    L = synth.make_layer(300 + H, 700, H, D, 2, xd, wd)
    dy = synth.make_x(301, 700, H, dyd)
    bounded_case(fff_lib, f"{xd}/{wd}/{dyd}/{dxd} H={H}", L, D, 2, dy, dx_dtype=dxd)


@pytest.mark.parametrize("act", ["gelu", "gelu_tanh", "identity"])
def test_bounded_activations(fff_lib, act):
    L = synth.make_layer(310, 2000, 768, 11, 1, "f32", "bf16")
    bounded_case(fff_lib, act, L, 11, 1, synth.make_x(311, 2000, 768, "f32"), act=act)


@pytest.mark.parametrize("H,wd", [(100, "f32"), (36, "bf16"), (2048, "bf16")])
def test_bounded_generic_widths(fff_lib, H, wd):
    L = synth.make_layer(320 + H, 500, H, 7, 3, wd, wd)
    bounded_case(fff_lib, f"generic H={H}", L, 7, 3, synth.make_x(321, 500, H, "f32"))


@pytest.mark.parametrize("B,D,T", [(1, 11, 1), (5, 3, 2), (257, 14, 1), (400, 15, 1), (300, 16, 1), (3000, 0, 64),
                                   (1000, 2, 300)])
def test_bounded_shapes(fff_lib, B, D, T):
    L = synth.make_layer(330 + B, B, 768, D, T, "bf16", "bf16")
    bounded_case(fff_lib, f"B={B} D={D} T={T}", L, D, T, synth.make_x(331, B, 768, "bf16"))


def test_device_forward_records_feed_the_backward(fff_lib):
    L = synth.make_layer(340, 5000, 768, 11, 1, "bf16", "bf16")
    bounded_case(fff_lib, "device path", L, 11, 1, synth.make_x(341, 5000, 768, "bf16"), path_from="device")


def test_accumulate_adds(fff_lib):
    L = synth.make_layer(350, 1500, 768, 8, 2, "f32", "f32")
    dy = synth.make_x(351, 1500, 768, "f32")
    fwd = oracle.forward(L["x"], L["w_in"], L["w_out"], 8, 2)
    leaves, lg = fwd["nodes"][:, :, 8].astype(np.int32), fwd["logits"].astype(np.float32)
    first = run_bwd(fff_lib, L, 8, 2, dy, leaves, lg)
    both = run_bwd(fff_lib, L, 8, 2, dy, leaves, lg, accumulate=True, init=first)
    assert np.array_equal(both["dx"], first["dx"] * 2)  # x + x is exact
    for k in ("dw_in", "dw_out"):
        scale = np.abs(first[k]).max()
        assert np.abs(both[k] - 2 * first[k]).max() <= 1e-5 * scale


def test_out_of_range_leaves_are_skipped_and_counted(fff_lib):
    B, H, D, T = 600, 768, 6, 2
    L = synth.make_layer(360, B, H, D, T, "f32", "f32")
    dy = synth.make_x(361, B, H, "f32")
    fwd = oracle.forward(L["x"], L["w_in"], L["w_out"], D, T)
    leaves = fwd["nodes"][:, :, D].astype(np.int32)
    bad_idx = [(3, 0, -1), (10, 1, 5), (599, 0, 2 ** (D + 1) - 1), (42, 1, 2 ** 30)]
    for b, t, v in bad_idx:
        leaves[b, t] = v
    bad = torch.zeros(1, dtype=torch.int32, device=DEV)
    got = run_bwd(fff_lib, L, D, T, dy, leaves, fwd["logits"].astype(np.float32), bad=bad)
    assert int(bad.item()) == len(bad_idx)
    # reference: per tree, the oracle over the tokens whose leaf in that tree is valid
    wshape = L["w_in"].shape
    ref = {"dx": np.zeros((B, H)), "dw_in": np.zeros(wshape), "dw_out": np.zeros(wshape)}
    for t in range(T):
        keep = np.array([not any(b == bb and t == tt for bb, tt, _ in bad_idx) for b in range(B)])
        r = oracle.backward(L["x"][keep], L["w_in"][t:t + 1], L["w_out"][t:t + 1], D, 1, dy[keep],
                            fwd["nodes"][keep][:, t:t + 1])
        ref["dx"][keep] += r["dx"]
        ref["dw_in"][t] = r["dw_in"][0]
        ref["dw_out"][t] = r["dw_out"][0]
    for k in ("dx", "dw_in", "dw_out"):
        err = np.abs(got[k] - ref[k]).max()
        assert err <= 1e-5 * np.abs(ref[k]).max(), (k, err)


def test_headline_layer_full_size(fff_lib):
    """65536 tokens, depth 11, bf16: the device forward's records through the backward, vs the oracle."""
    from paper_2311_10770_amd.configs import WORKLOADS

    w = WORKLOADS["d11_h768_b65536_bf16"]
    L = synth.make_layer(w.seed, w.n_tokens, w.hidden, w.depth, w.n_trees, w.x_dtype, w.w_dtype)
    bounded_case(fff_lib, "d11 65536 bf16", L, w.depth, w.n_trees, synth.make_x(w.seed + 100, w.n_tokens,
                                                                                   w.hidden, "bf16"),
                 path_from="device", dx_dtype="bf16")


@pytest.mark.parametrize("B,H,D", [(6000, 768, 11), (5000, 1024, 9)])
def test_bitwise_reproducible_with_skewed_and_one_hot_leaves(fff_lib, B, H, D):
    """Two backward calls on the same inputs give the same bits (no atomics, stable leaf order, fixed
    summation order), with clustered tokens (skewed leaves) and with every token on one path (a
    single leaf holding the whole batch, more token ids than one workgroup stages in LDS)."""
    for kind in ("clustered", "one path"):
        if kind == "clustered":
            x = synth.make_clustered_x(360 + H, B, H, "bf16")
        else:
            x = np.repeat(synth.make_x(361 + H, 1, H, "bf16"), B, axis=0)
        wi, wo = synth.make_weights(360 + H, H, D, 1, "bf16")
        L = {"x": x, "w_in": wi, "w_out": wo}
        dy = synth.make_x(362 + H, B, H, "bf16")
        fwd = oracle.forward(x, wi, wo, D, 1)
        leaves = fwd["nodes"][:, :, D].astype(np.int32)
        logits32 = fwd["logits"].astype(np.float32)
        flush_print(f"[gpu] bwd twice {kind}: B={B} H={H} D={D}, largest leaf {np.bincount(leaves[:, 0]).max()}")
        a = run_bwd(fff_lib, L, D, 1, dy, leaves, logits32)
        b = run_bwd(fff_lib, L, D, 1, dy, leaves, logits32)
        for k in ("dx", "dw_in", "dw_out"):
            assert np.array_equal(a[k].view(np.uint32), b[k].view(np.uint32)), (kind, k)
        ref = oracle.backward(x, wi, wo, D, 1, dy, fwd["nodes"])
        rep = parity.backward_check(x, wi, wo, D, 1, dy, fwd["nodes"], logits32, a, ref)
        assert rep["ok"], (kind, rep["fail"])


@pytest.mark.parametrize("xd,dyd,H", [("bf16", "f32", 640), ("f32", "bf16", 128), ("bf16", "bf16", 256)])
def test_fused_types_and_widths(fff_lib, xd, dyd, H):
    """The fused leaf-tiled path (one tree, bf16 W, hidden a multiple of 128 up to 1024) with the x / dy
    type pairs and workgroup sizes the other cases leave out: 5 waves (three of them alone on a SIMD
    compute the tile's activations), 1 wave and 2 waves."""
    D = 9
    L = synth.make_layer(370 + H, 900, H, D, 1, xd, "bf16")
    bounded_case(fff_lib, f"fused {xd}/{dyd} H={H}", L, D, 1, synth.make_x(371 + H, 900, H, dyd))


def test_fused_accumulate_dw_only_and_bad_leaves(fff_lib):
    """On the fused path: accumulation doubles every output, dW alone (no dx requested) equals the dW
    of a full call bit for bit, and out-of-range leaves are counted and get zero dx rows while the
    other tokens match the oracle."""
    B, H, D = 3000, 768, 10
    L = synth.make_layer(380, B, H, D, 1, "bf16", "bf16")
    dy = synth.make_x(381, B, H, "bf16")
    fwd = oracle.forward(L["x"], L["w_in"], L["w_out"], D, 1)
    leaves, lg = fwd["nodes"][:, :, D].astype(np.int32), fwd["logits"].astype(np.float32)
    first = run_bwd(fff_lib, L, D, 1, dy, leaves, lg)
    both = run_bwd(fff_lib, L, D, 1, dy, leaves, lg, accumulate=True, init=first)
    assert np.array_equal(both["dx"], first["dx"] * 2)  # x + x is exact
    for k in ("dw_in", "dw_out"):
        assert np.abs(both[k] - 2 * first[k]).max() <= 1e-5 * np.abs(first[k]).max(), k
    _, dwi, dwo = fff_lib.backward(dev(fff_lib, L["x"]), dev(fff_lib, L["w_in"]), dev(fff_lib, L["w_out"]), D, 1,
                                   dev(fff_lib, dy), dev(fff_lib, leaves), dev(fff_lib, lg), act="gelu",
                                   want=("dw_in", "dw_out"))
    torch.cuda.synchronize()
    assert np.array_equal(fff_lib.to_numpy(dwi).view(np.uint32), first["dw_in"].view(np.uint32))
    assert np.array_equal(fff_lib.to_numpy(dwo).view(np.uint32), first["dw_out"].view(np.uint32))
    bad_rows = [0, 17, 1500, B - 1]
    bad_leaves = leaves.copy()
    for i, b in enumerate(bad_rows):
        bad_leaves[b, 0] = [-1, 5, 2 ** (D + 1) - 1, 2 ** 30][i]
    bad = torch.zeros(1, dtype=torch.int32, device=DEV)
    got = run_bwd(fff_lib, L, D, 1, dy, bad_leaves, lg, bad=bad)
    assert int(bad.item()) == len(bad_rows)
    assert not got["dx"][bad_rows].any()
    keep = np.ones(B, dtype=bool)
    keep[bad_rows] = False
    ref = oracle.backward(L["x"][keep], L["w_in"], L["w_out"], D, 1, dy[keep], fwd["nodes"][keep])
    for k in ("dx", "dw_in", "dw_out"):
        g = got[k][keep] if k == "dx" else got[k]
        err = np.abs(g - ref[k]).max()
        assert err <= 1e-5 * np.abs(ref[k]).max(), (k, err)
