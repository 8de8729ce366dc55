"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Paths must match the oracle node for node except after a flagged near tie;
outputs must meet the per-token normwise bar (1e-5 for fp32 outputs, 2e-2
for bf16 outputs), evaluated along the device's own path.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import parity
from paper_2311_10770_amd import synth
from paper_2311_10770_amd.configs import WORKLOADS
from tests.conftest import flush_print
from tests.gpu_util import DEV, TORCH_DT, check_layer, layer, run_fff, tol_for

pytestmark = pytest.mark.gpu


# ------------------------------------------------------------ named workloads


@pytest.mark.parametrize("name", ["d3_h768_b128_f32", "d11_h768_b16384_f32", "d11_h768_b65536_bf16",
                                  "d11_h768_b65536_w_bf16", "4x9_h768_b16384_f32", "4x8_h768_b16384_f32"])
def test_workload_full_size(fff_lib, name):
    w = WORKLOADS[name]
    L = synth.make_layer(w.seed, w.n_tokens, w.hidden, w.depth, w.n_trees, w.x_dtype, w.w_dtype)
    check_layer(fff_lib, name, L, w.depth, w.n_trees, w.y_dtype)


def test_llm_width_tree_batch_sweep(fff_lib):
    """Depth 15 (65535 nodes) at hidden 4096, bf16; smaller batches are prefixes of the largest draw."""
    w = WORKLOADS["d15_h4096_bf16"]
    L = synth.make_layer(w.seed, max(w.sweep), w.hidden, w.depth, w.n_trees, w.x_dtype, w.w_dtype)
    for B in w.sweep:
        Lb = dict(L, x=L["x"][:B])
        check_layer(fff_lib, f"d15_h4096 B={B}", Lb, w.depth, w.n_trees, w.y_dtype)


def test_stacked_layers_teacher_forced(fff_lib):
    """Twelve 4x9 layers with x <- x + FFF(x); each layer is checked on the device's own input."""
    w = WORKLOADS["4x9_h768_b16384_f32_x12"]
    B = 4096
    x = synth.make_x(w.seed, B, w.hidden, "f32")
    for layer_idx in range(w.layers):
        wi, wo = synth.make_weights(w.seed, w.hidden, w.depth, w.n_trees, "f32", layer=layer_idx + 1)
        L = {"x": x, "w_in": wi, "w_out": wo}
        got = run_fff(fff_lib, L, w.depth, w.n_trees, "f32", out="residual")
        ref = oracle.forward(x, wi, wo, w.depth, w.n_trees)
        parity.assert_parity(x, wi, wo, w.depth, w.n_trees, ref, got["y"], got["nodes"], tol=1e-5, base_dev=x)
        x = got["y"].astype(np.float32)


# ------------------------------------------------ the KxD family of Table 1

from paper_2311_10770_amd.configs import KXD_FAMILY  # noqa: E402


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("k,d", KXD_FAMILY)
def test_kxd_family(fff_lib, k, d, dtype):
    """Every UltraFastBERT-KxD shape through the default plan, 131 tokens (ragged)."""
    L = layer(6, 131, 768, d, k, dtype, dtype)
    check_layer(fff_lib, f"{k}x{d} {dtype}", L, d, k, dtype)


# ------------------------------------------------------ shapes, dtypes, edges

DTYPE_COMBOS = [("f32", "f32", "f32"), ("bf16", "bf16", "bf16"), ("f32", "bf16", "f32"), ("bf16", "bf16", "f32"),
                ("bf16", "f32", "f32"), ("f32", "f32", "bf16"), ("f32", "bf16", "bf16"), ("bf16", "f32", "bf16")]


@pytest.mark.parametrize("xd,wd,yd", DTYPE_COMBOS)
@pytest.mark.parametrize("H", [768, 1024, 4096])
def test_dtype_combinations_fast_widths(fff_lib, xd, wd, yd, H):
    depth = 6 if H == 4096 else 8
    L = layer(20 + H, 777, H, depth, 1, xd, wd)
    check_layer(fff_lib, f"{xd}/{wd}/{yd} H={H}", L, depth, 1, yd)


@pytest.mark.parametrize("B", [1, 2, 3, 4, 5, 63, 64, 65, 255, 257, 1000, 4097])
def test_ragged_token_counts(fff_lib, B):
    L = layer(30, B, 768, 11, 1, "bf16", "bf16")
    check_layer(fff_lib, f"ragged B={B}", L, 11, 1, "bf16")


@pytest.mark.parametrize("H", [1, 2, 8, 63, 100, 767, 769, 1536, 2048])
@pytest.mark.parametrize("wd", ["f32", "bf16"])
def test_generic_hidden_sizes(fff_lib, H, wd):
    L = layer(40 + H, 200, H, 5, 2, wd, wd)
    check_layer(fff_lib, f"generic H={H} w={wd}", L, 5, 2, "f32")


@pytest.mark.parametrize("depth,trees", [(0, 1), (0, 64), (1, 3), (11, 4), (14, 1), (2, 300)])
def test_depth_and_tree_edges(fff_lib, depth, trees):
    """Depth 0 with one tree is a single neuron, y = act(l) W_out[0]: a token whose logit nearly
    cancels (|l| far below sum_i |x_i W_in[0, i]|) is ill-conditioned in the checker's sense and may
    use its rounding allowance; everywhere else the raw 1e-5 bar holds."""
    L = layer(50 + depth, 300, 768, depth, trees, "f32", "f32")
    check_layer(fff_lib, f"depth={depth} trees={trees}", L, depth, trees, "f32",
                max_conditioned=300 if (depth, trees) == (0, 1) else 0)


@pytest.mark.parametrize("mode", ["descent", "generic", "grouped"])
def test_modes_agree(fff_lib, mode):
    L = layer(60, 3000, 768, 11, 2, "f32", "bf16")
    check_layer(fff_lib, f"mode={mode}", L, 11, 2, "f32", mode=mode)


# --------------------------------------------------------------- grouped mode


@pytest.mark.parametrize("name", ["d11_h768_b65536_bf16", "d11_h768_b16384_f32", "4x9_h768_b16384_f32"])
def test_grouped_full_size(fff_lib, name):
    w = WORKLOADS[name]
    L = synth.make_layer(w.seed, w.n_tokens, w.hidden, w.depth, w.n_trees, w.x_dtype, w.w_dtype)
    check_layer(fff_lib, f"grouped {name}", L, w.depth, w.n_trees, w.y_dtype, mode="grouped")


@pytest.mark.parametrize("split", [-1, 0, 3, 4, 6, 11])
@pytest.mark.parametrize("B", [1, 7, 1000, 5003])
def test_grouped_split_levels_and_ragged(fff_lib, split, B):
    L = layer(160 + B, B, 768, 11, 1, "bf16", "bf16")
    check_layer(fff_lib, f"grouped split={split} B={B}", L, 11, 1, "bf16", mode="grouped", split_level=split)


@pytest.mark.parametrize("xd,wd,yd", DTYPE_COMBOS)
@pytest.mark.parametrize("H", [768, 1024, 4096])
def test_grouped_dtype_combinations(fff_lib, xd, wd, yd, H):
    depth = 6 if H == 4096 else 9
    L = layer(170 + H, 900, H, depth, 2, xd, wd)
    check_layer(fff_lib, f"grouped {xd}/{wd}/{yd} H={H}", L, depth, 2, yd, mode="grouped")


def test_grouped_matches_descent_bitwise(fff_lib):
    """Same per-token arithmetic in the same order: the two modes agree bit for bit."""
    L = layer(180, 20000, 768, 11, 1, "bf16", "bf16")
    a = run_fff(fff_lib, L, 11, 1, "bf16", mode="descent")
    b = run_fff(fff_lib, L, 11, 1, "bf16", mode="grouped")
    assert np.array_equal(a["y"], b["y"]) and np.array_equal(a["nodes"], b["nodes"])
    assert np.array_equal(a["logits"], b["logits"])


def test_grouped_out_modes_and_skewed_routing(fff_lib):
    B = 6000
    x = synth.make_clustered_x(190, B, 768, "f32")
    wi, wo = synth.make_weights(190, 768, 11, 1, "f32")
    L = {"x": x, "w_in": wi, "w_out": wo}
    ref = oracle.forward(x, wi, wo, 11, 1)
    res = run_fff(fff_lib, L, 11, 1, "f32", mode="grouped", out="residual")
    parity.assert_parity(x, wi, wo, 11, 1, ref, res["y"], res["nodes"], tol=1e-5, base_dev=x)
    y0 = synth.make_x(191, B, 768, "f32")
    acc = run_fff(fff_lib, L, 11, 1, "f32", y_init=y0, mode="grouped", out="accumulate")
    parity.assert_parity(x, wi, wo, 11, 1, ref, acc["y"], acc["nodes"], tol=1e-5, base_dev=y0)


def test_grouped_workspace_errors(fff_lib):
    L = layer(200, 512, 768, 11, 1, "bf16", "bf16")
    x, wi, wo = (fff_lib.from_numpy(L[k], DEV) for k in ("x", "w_in", "w_out"))
    need = fff_lib.workspace_bytes(512, 11, 1, 768)  # covers grouped and tiled mode
    grouped_need = 512 * 12 * 4 + 512 * 4  # activation records and leaves, each a multiple of 256 bytes
    assert need > grouped_need
    for mode, n in (("grouped", grouped_need), ("tiled", need)):
        small = torch.empty(n - 256, dtype=torch.uint8, device=DEV)
        with pytest.raises(fff_lib.FffError) as e:
            fff_lib.forward(x, wi, wo, 11, 1, mode=mode, workspace=small)
        assert e.value.status == fff_lib.fff.FFF_ERR_WORKSPACE
    big = torch.empty(need + 4096, dtype=torch.uint8, device=DEV)
    with pytest.raises(fff_lib.FffError) as e:
        fff_lib.forward(x, wi, wo, 11, 1, mode="grouped", workspace=big[16:])  # misaligned
    assert e.value.status == fff_lib.fff.FFF_ERR_WORKSPACE
    with pytest.raises(fff_lib.FffError):
        fff_lib.forward(x, wi, wo, 11, 1, mode="grouped", split_level=2)  # fewer subtrees than XCDs


@pytest.mark.parametrize("lds_levels", [-1, 1, 3, 5])
def test_lds_levels_do_not_change_bits(fff_lib, lds_levels):
    L = layer(70, 2000, 768, 11, 1, "bf16", "bf16")
    base = run_fff(fff_lib, L, 11, 1, "f32", lds_levels=-1)
    got = run_fff(fff_lib, L, 11, 1, "f32", lds_levels=lds_levels)
    assert np.array_equal(base["y"], got["y"]) and np.array_equal(base["nodes"], got["nodes"])


def test_activation_variants(fff_lib):
    L = layer(80, 500, 768, 9, 1, "f32", "f32")
    check_layer(fff_lib, "gelu_tanh", L, 9, 1, "f32", act="gelu_tanh")
    check_layer(fff_lib, "identity", L, 9, 1, "f32", act="identity")


@pytest.mark.parametrize("act", ["gelu_tanh", "identity"])
def test_activation_variants_masked_and_subtree(fff_lib, act):
    L = layer(81, 300, 768, 3, 16, "bf16", "bf16")
    check_layer(fff_lib, f"masked {act}", L, 3, 16, "f32", act=act, mode="masked")
    L = layer(82, 40, 768, 9, 2, "f32", "f32")
    check_layer(fff_lib, f"subtree {act}", L, 9, 2, "f32", act=act, mode="subtree")


@pytest.mark.parametrize("H,mode,T,wd", [(768, "descent", 2, "f32"), (40, "generic", 2, "f32"),
                                         (768, "subtree", 2, "f32"), (768, "masked", 2, "f32"),
                                         (768, "grouped", 2, "f32"), (768, "grouped", 1, "bf16"),
                                         (768, "tiled", 1, "f32"), (768, "tiled", 1, "bf16")])
def test_small_integers_identity_bit_exact_with_ties(fff_lib, H, mode, T, wd):
    """Identity activation on small integers: every value is an exact integer, so the device
    must match the oracle bit for bit, including logits of exactly zero (they go left).  bf16
    weights and x hold the same integers exactly; the leaf-tiled MFMA emit splits each integer
    activation into bf16 parts that sum to it exactly."""
    D, B = 6, 300
    L = synth.small_int_layer(9, B, H, D, T)
    for b in range(0, B, 5):  # exact zero at the root of tree 0
        w0 = L["w_in"][0, 0]
        i, j = np.nonzero(w0)[0][:2]
        L["x"][b] = 0
        L["x"][b, i], L["x"][b, j] = w0[j], -w0[i]
    if wd == "bf16":
        L = {k: synth.as_dtype(v, "bf16") for k, v in L.items()}
    got = run_fff(fff_lib, L, D, T, "f32", act="identity", mode=mode)
    ref = oracle.forward(L["x"], L["w_in"], L["w_out"], D, T, act="identity")
    assert np.array_equal(got["nodes"], ref["nodes"])
    assert np.array_equal(got["y"].astype(np.float64), ref["y"])
    assert np.all(got["nodes"][::5, 0, 1] == 1)


def test_device_gelu_on_a_dense_grid(fff_lib):
    """The device activation itself (P7): a depth-0 tree with W_in = W_out = e_0 and x[b, 0] = z_b
    gives y[b] = act(z_b) e_0 exactly (the logit is z_b, the output a product by 1), so y[:, 0] is the
    kernels' GELU on a grid of 36001 points in [-9, 9], compared with the fp64 GELU in units of the
    fp32 unit roundoff u.  Exact form z/2 erfc(-z/sqrt 2): the argument is formed in fp32 (the
    rounded constant and one product: relative error below 1.3 u), which erfc's condition number
    (about z^2 + 1) magnifies; erfcf's own error is a few ulp (8 u) and the final product one more
    rounding: bound (11 + 1.3 (z^2 + 1)) u.  Tanh form z / (1 + exp(-2v)), v = sqrt(2/pi)(z +
    0.044715 z^3): v carries about 3 u of relative error, which exp magnifies by |2v|: bound
    (11 + 6 |v|) u.  Between -3 and 3 both stay within a few ulp.  The other columns must be
    exactly 0.  Both forms, through every mode with a depth-0 kernel."""
    z = np.linspace(-9.0, 9.0, 36001).astype(np.float32)
    H = 768
    x = np.zeros((z.size, H), dtype=np.float32)
    x[:, 0] = z
    e0 = np.zeros((1, 1, H), dtype=np.float32)
    e0[0, 0, 0] = 1.0
    L = {"x": x, "w_in": e0, "w_out": e0.copy()}
    zd = z.astype(np.float64)
    for act in ("gelu", "gelu_tanh"):
        want = parity.act_values(zd, act)
        for mode in ("descent", "generic", "masked", "subtree"):
            got = run_fff(fff_lib, L, 0, 1, "f32", act=act, mode=mode, record=False)["y"]
            assert np.all(got[:, 1:] == 0.0), mode
            err = np.abs(got[:, 0].astype(np.float64) - want)
            if act == "gelu":
                units = 11.0 + 1.3 * (zd * zd + 1.0)
            else:
                units = 11.0 + 6.0 * np.abs(np.sqrt(2.0 / np.pi) * (zd + 0.044715 * zd ** 3))
            bound = units * 2.0 ** -24 * np.abs(want) + 1e-45
            worst = int(np.argmax(err / bound))
            assert np.all(err <= bound), f"{act} {mode}: z={zd[worst]} got {got[worst, 0]!r} want {want[worst]!r}"
            mid = np.abs(zd) <= 3.0
            ulps = float((err[mid] / (2.0 ** -23 * np.abs(want[mid]) + 1e-45)).max())
            flush_print(f"[gpu] gelu grid {act} {mode}: max err/bound {float((err / bound).max()):.3f}, "
                        f"max {ulps:.2f} ulp on [-3, 3]")


def test_out_modes(fff_lib):
    L = layer(90, 1500, 768, 10, 1, "f32", "f32")
    y0 = synth.make_x(91, 1500, 768, "f32")
    ref = oracle.forward(L["x"], L["w_in"], L["w_out"], 10, 1)
    acc = run_fff(fff_lib, L, 10, 1, "f32", y_init=y0, out="accumulate")
    parity.assert_parity(L["x"], L["w_in"], L["w_out"], 10, 1, ref, acc["y"], acc["nodes"], tol=1e-5, base_dev=y0)
    res = run_fff(fff_lib, L, 10, 1, "f32", out="residual")
    parity.assert_parity(L["x"], L["w_in"], L["w_out"], 10, 1, ref, res["y"], res["nodes"], tol=1e-5,
                         base_dev=L["x"])


def test_plain_six_argument_entry_point(fff_lib):
    L = layer(100, 999, 768, 11, 1, "bf16", "bf16")
    x, wi, wo = (fff_lib.from_numpy(L[k], DEV) for k in ("x", "w_in", "w_out"))
    y = torch.empty((999, 768), dtype=torch.bfloat16, device=DEV)
    fff_lib.forward_plain(x, wi, wo, 11, 1, y)
    torch.cuda.synchronize()
    ref = oracle.forward(L["x"], L["w_in"], L["w_out"], 11, 1)
    parity.assert_parity(L["x"], L["w_in"], L["w_out"], 11, 1, ref, fff_lib.to_numpy(y), None, tol=2e-2)


# ------------------------------------------------- determinism, streams, guards


@pytest.mark.parametrize("case", ["descent", "tiled_headline", "tiled_spills", "grouped"])
def test_deterministic(fff_lib, case):
    """Two runs give the same bits: the fused kernel, the leaf-tiled path at the headline size (its
    bucket slots are taken by atomics in any order), the leaf-tiled path with clustered tokens that
    overflow their buckets, and the grouped path."""
    if case == "tiled_headline":
        w = WORKLOADS["d11_h768_b65536_bf16"]
        L = synth.make_layer(w.seed, w.n_tokens, w.hidden, w.depth, w.n_trees, w.x_dtype, w.w_dtype)
        mode = "auto"
        x, wi, wo = (fff_lib.from_numpy(L[k], DEV) for k in ("x", "w_in", "w_out"))
        assert fff_lib.describe(x, wi, wo, 11, 1).startswith("tiled<")
    elif case == "tiled_spills":
        x = synth.make_clustered_x(111, 20000, 768, "bf16", n_centres=8)
        wi, wo = synth.make_weights(111, 768, 11, 1, "bf16")
        L, mode = {"x": x, "w_in": wi, "w_out": wo}, "tiled"
    else:
        L, mode = layer(110, 20000, 768, 11, 1, "bf16", "bf16"), case
    flush_print(f"[gpu] deterministic {case}")
    runs = [run_fff(fff_lib, L, 11, 1, "bf16", mode=mode) for _ in range(3)]
    for r in runs[1:]:
        assert np.array_equal(runs[0]["y"], r["y"]) and np.array_equal(runs[0]["nodes"], r["nodes"])
        assert np.array_equal(runs[0]["logits"], r["logits"])


def test_non_default_stream(fff_lib):
    L = layer(120, 4000, 768, 11, 1, "f32", "f32")
    x, wi, wo = (fff_lib.from_numpy(L[k], DEV) for k in ("x", "w_in", "w_out"))
    s = torch.cuda.Stream(device=DEV)
    y = torch.empty((4000, 768), dtype=torch.float32, device=DEV)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        fff_lib.forward(x, wi, wo, 11, 1, y)
    s.synchronize()
    ref = oracle.forward(L["x"], L["w_in"], L["w_out"], 11, 1)
    parity.assert_parity(L["x"], L["w_in"], L["w_out"], 11, 1, ref, y.cpu().numpy(), None, tol=1e-5)


@pytest.mark.parametrize("yd,mode", [("bf16", "descent"), ("f32", "descent"), ("f32", "generic"),
                                     ("bf16", "tiled"), ("f32", "tiled"), ("bf16", "grouped"), ("f32", "grouped"),
                                     ("bf16", "masked"), ("f32", "subtree")])
def test_guard_bands_untouched(fff_lib, yd, mode):
    """No kernel writes outside y and the records: both are placed between bands of sentinels (the
    masked mode at depth 5, the others at depth 11; 517 tokens, a ragged count)."""
    B, H = 517, 768
    D = 5 if mode == "masked" else 11
    L = layer(130, B, H, D, 1, "bf16", "bf16")
    x, wi, wo = (fff_lib.from_numpy(L[k], DEV) for k in ("x", "w_in", "w_out"))
    pad = 4096
    buf = torch.full((B * H + 2 * pad,), 12345.0, dtype=TORCH_DT[yd], device=DEV)
    y = buf[pad:pad + B * H].view(B, H)
    nbuf = torch.full((B * (D + 1) + 2 * pad,), -99, dtype=torch.int32, device=DEV)
    nodes = nbuf[pad:pad + B * (D + 1)]
    lbuf = torch.full((B * (D + 1) + 2 * pad,), 777.0, dtype=torch.float32, device=DEV)
    logits = lbuf[pad:pad + B * (D + 1)]
    fff_lib.forward(x, wi, wo, D, 1, y, nodes_out=nodes, logits_out=logits, mode=mode)
    torch.cuda.synchronize()
    assert torch.all(buf[:pad] == 12345.0) and torch.all(buf[-pad:] == 12345.0)
    assert torch.all(nbuf[:pad] == -99) and torch.all(nbuf[-pad:] == -99)
    assert torch.all(lbuf[:pad] == 777.0) and torch.all(lbuf[-pad:] == 777.0)
    ref = oracle.forward(L["x"], L["w_in"], L["w_out"], D, 1)
    parity.assert_parity(L["x"], L["w_in"], L["w_out"], D, 1, ref, fff_lib.to_numpy(y), nodes.view(B, 1, D + 1)
                         .cpu().numpy(), tol=tol_for("bf16", yd))


def test_describe_names_the_kernel(fff_lib):
    L = layer(140, 64, 768, 11, 1, "bf16", "bf16")
    x, wi, wo = (fff_lib.from_numpy(L[k], DEV) for k in ("x", "w_in", "w_out"))
    d = fff_lib.describe(x, wi, wo, 11, 1)  # auto, 64 tokens: a workgroup per token
    assert d.startswith("subtree<"), d
    xm = torch.zeros((1024, 768), dtype=torch.bfloat16, device=DEV)
    d = fff_lib.describe(xm, wi, wo, 11, 1)  # auto, 1024 tokens: the fused kernel
    assert d.startswith("descent<"), d
    xf = torch.zeros((16384, 768), dtype=torch.float32, device=DEV)
    wf = torch.zeros((1, (1 << 12) - 1, 768), dtype=torch.float32, device=DEV)
    assert fff_lib.describe(xf, wf, wf, 11, 1).startswith("tiled<")  # fp32, 16384 tokens: 8 per leaf
    assert fff_lib.describe(xf[:8192], wf, wf, 11, 1).startswith("descent<")  # 4 per leaf, 6.3M elements
    for d, B, want in ((12, 16384, "tiled<"), (13, 16384, "tiled<"), (14, 32768, "tiled<"), (14, 16384, "grouped<")):
        xfd = torch.zeros((B, 768), dtype=torch.float32, device=DEV)  # fp32 leaf pairs from 2 per leaf, 12M
        wfd = torch.zeros((1, (2 << d) - 1, 768), dtype=torch.float32, device=DEV)
        assert fff_lib.describe(xfd, wfd, wfd, d, 1).startswith(want), (d, B)
        del xfd, wfd
    xw = torch.zeros((8192, 4096), dtype=torch.bfloat16, device=DEV)
    ww = torch.zeros((1, (1 << 12) - 1, 4096), dtype=torch.bfloat16, device=DEV)
    assert fff_lib.describe(xw, ww, ww, 11, 1).startswith("tiled<")  # 4 per leaf, hidden 4096
    assert fff_lib.describe(xw[:4096], ww, ww, 11, 1).startswith("descent<")  # 2 per leaf
    del xw, ww
    w9 = torch.zeros((1, (1 << 10) - 1, 768), dtype=torch.bfloat16, device=DEV)
    xb9 = torch.zeros((32768, 768), dtype=torch.bfloat16, device=DEV)
    assert fff_lib.describe(xb9, w9, w9, 9, 1).startswith("descent<")  # bf16 depth 9, 32768 tokens
    xb9 = torch.zeros((131072, 768), dtype=torch.bfloat16, device=DEV)
    assert fff_lib.describe(xb9[:65536], w9, w9, 9, 1).startswith("descent<")  # 48M elements
    assert fff_lib.describe(xb9, w9, w9, 9, 1).startswith("tiled<")  # 96M elements
    del xb9
    xf5 = torch.zeros((65536, 768), dtype=torch.float32, device=DEV)
    wf5 = torch.zeros((1, 63, 768), dtype=torch.float32, device=DEV)
    assert fff_lib.describe(xf5, wf5, wf5, 5, 1).startswith("grouped<")  # fp32 depth 5, 65536 tokens
    assert fff_lib.describe(xf5[:32768], wf5, wf5, 5, 1).startswith("descent<")
    # auto with the binding's workspace at 64K tokens: leaf tiles at 32 tokens per leaf,
    # subtree grouping at 4 per leaf (planning only: nothing is launched)
    xb = torch.zeros((65536, 768), dtype=torch.bfloat16, device=DEV)
    assert fff_lib.describe(xb, wi, wo, 11, 1).startswith("tiled<")
    assert fff_lib.describe(xb[:32768], wi, wo, 11, 1).startswith("tiled<")  # 16 per leaf, 25M elements
    assert fff_lib.describe(xb[:16384], wi, wo, 11, 1).startswith("descent<")  # 8 per leaf, 12.6M
    w14 = torch.zeros((1, (1 << 15) - 1, 768), dtype=torch.bfloat16, device=DEV)
    assert fff_lib.describe(xb, w14, w14, 14, 1).startswith("grouped<")
    d = fff_lib.describe(x, wi, wo, 11, 1, mode="descent")
    assert d.startswith("descent<") and "lds_levels=" in d
    wi4 = fff_lib.from_numpy(np.concatenate([L["w_in"]] * 4), DEV)
    assert fff_lib.describe(xm, wi4, wi4, 11, 4).startswith("descent<")  # several trees: fused kernel
    assert fff_lib.describe(x, wi4, wi4, 11, 4).startswith("subtree<")  # 64 tokens x 4 trees
    d = fff_lib.describe(x, wi, wo, 11, 1, mode="generic")
    assert d.startswith("generic")
    d = fff_lib.describe(x, wi, wo, 11, 1, mode="grouped")
    assert d.startswith("grouped<") and "split_level=5" in d and "launch1" in d


def test_errors_surface_as_exceptions(fff_lib):
    L = layer(150, 16, 768, 3, 1, "f32", "f32")
    x, wi, wo = (fff_lib.from_numpy(L[k], DEV) for k in ("x", "w_in", "w_out"))
    with pytest.raises(fff_lib.FffError):
        fff_lib.forward(x, wi, wo, 3, 1, lds_levels=9)  # more levels than the tree has
    with pytest.raises(ValueError):
        fff_lib.forward(x, wi[:, :7], wo, 3, 1)
    buf = torch.zeros(17 * 768, device=DEV)
    xb = buf[:16 * 768].view(16, 768)
    xb.copy_(x)
    with pytest.raises(fff_lib.FffError):
        fff_lib.forward(xb, wi, wo, 3, 1, y=buf[768:].view(16, 768))  # y overlaps x without being x
    with pytest.raises(fff_lib.FffError):
        fff_lib.forward(x[:8], wi, wo, 3, 1, y=wi.view(-1)[:8 * 768].view(8, 768))  # y overlaps W_in


# ----------------------------------------------------------------- tiled mode


@pytest.mark.parametrize("xd,wd,yd", DTYPE_COMBOS)
@pytest.mark.parametrize("H", [768, 1024, 4096])
def test_tiled_dtype_combinations(fff_lib, xd, wd, yd, H):
    depth = 7 if H == 4096 else 9
    L = layer(190 + H, 1500, H, depth, 1, xd, wd)
    check_layer(fff_lib, f"tiled {xd}/{wd}/{yd} H={H}", L, depth, 1, yd, mode="tiled")


@pytest.mark.parametrize("B", [1, 7, 100, 2049, 30001])
@pytest.mark.parametrize("depth", [5, 8, 11, 15])
def test_tiled_ragged_and_depths(fff_lib, B, depth):
    L = layer(200 + B + depth, B, 768, depth, 1, "bf16", "bf16")
    check_layer(fff_lib, f"tiled B={B} D={depth}", L, depth, 1, "bf16", mode="tiled")


@pytest.mark.parametrize("out", ["residual", "accumulate"])
def test_tiled_output_modes(fff_lib, out):
    L = layer(210, 3000, 768, 11, 1, "f32", "f32")
    y0 = synth.make_x(211, 3000, 768, "f32")
    got = run_fff(fff_lib, L, 11, 1, "f32", mode="tiled", out=out, y_init=y0 if out == "accumulate" else None)
    ref = oracle.forward(L["x"], L["w_in"], L["w_out"], 11, 1)
    base = L["x"] if out == "residual" else y0
    parity.assert_parity(L["x"], L["w_in"], L["w_out"], 11, 1, ref, got["y"], got["nodes"], tol=1e-5,
                         base_dev=base)


def test_tiled_skewed_routing_spills(fff_lib):
    """Clustered tokens crowd a few leaves: most of them overflow their bucket and take the spill path."""
    B, H, D = 20000, 768, 11
    x = synth.make_clustered_x(220, B, H, "bf16", n_centres=8)
    wi, wo = synth.make_weights(220, H, D, 1, "bf16")
    check_layer(fff_lib, "tiled clustered", {"x": x, "w_in": wi, "w_out": wo}, D, 1, "bf16", mode="tiled")


def test_tiled_headline_full_size(fff_lib):
    w = WORKLOADS["d11_h768_b65536_bf16"]
    L = synth.make_layer(w.seed, w.n_tokens, w.hidden, w.depth, w.n_trees, w.x_dtype, w.w_dtype)
    check_layer(fff_lib, "tiled headline", L, w.depth, w.n_trees, w.y_dtype, mode="tiled")


@pytest.mark.parametrize("case", ["bf16_2trees_store", "f32_residual"])
def test_tiled_token_chunks(fff_lib, case):
    """A tiled call whose fp32 rows pass 2^31 bytes runs as consecutive token chunks of
    (2^31 - 1) / (4 H) tokens: 700000 tokens at H = 768 are 699050 + 4950.  Every output row is
    written (no NaN left, every node recorded); tokens at the start, on both sides of the seam
    and at the end match the oracle (two trees with a bf16 y: the fp32 running sum of each
    chunk; fp32 residual: the source rows of each chunk)."""
    B, H, D = 700000, 768, 11
    chunk = ((1 << 31) - 1) // (4 * H)
    T, dt, out = (2, "bf16", "store") if case == "bf16_2trees_store" else (1, "f32", "residual")
    x = synth.make_x(240, B, H, dt)
    wi, wo = synth.make_weights(240, H, D, T, dt)
    flush_print(f"[gpu] tiled token chunks {case}: B={B} chunk={chunk}")
    xd, wid, wod = (fff_lib.from_numpy(a, DEV) for a in (x, wi, wo))
    y = torch.full((B, H), float("nan"), dtype=TORCH_DT[dt], device=DEV)
    nodes = torch.full((B, T, D + 1), -7, dtype=torch.int32, device=DEV)
    assert fff_lib.describe(xd, wid, wod, D, T, mode="tiled", out=out).startswith("tiled<")
    fff_lib.forward(xd, wid, wod, D, T, y, nodes_out=nodes, mode="tiled", out=out)
    torch.cuda.synchronize()
    assert not bool(torch.isnan(y).any()) and bool((nodes >= 0).all())
    idx = np.r_[0:256, chunk - 256:chunk + 256, B - 256:B]
    it = torch.from_numpy(idx).to(DEV)
    got_y = fff_lib.to_numpy(y.index_select(0, it))
    got_nodes = nodes.index_select(0, it).cpu().numpy()
    del y, nodes, xd
    xs = x[idx]
    ref = oracle.forward(xs, wi, wo, D, T)
    parity.assert_parity(xs, wi, wo, D, T, ref, got_y, got_nodes, tol=tol_for(dt, dt),
                         base_dev=xs if out == "residual" else None)


@pytest.mark.parametrize("yd", ["f32", "bf16"])
def test_tiled_with_layernorm(fff_lib, yd):
    """The leaf-tiled path behind the LayerNorm prologue, with the residual: y = x + FFF(LN(x)),
    against the oracle's block on the device's own paths."""
    B = 5000
    L = layer(230, B, 768, 11, 1, "bf16", "bf16")
    gamma, beta = synth.make_norm(230, 768)
    x = fff_lib.from_numpy(L["x"], DEV)
    wi, wo = fff_lib.from_numpy(L["w_in"], DEV), fff_lib.from_numpy(L["w_out"], DEV)
    nodes = torch.empty((B, 1, 12), dtype=torch.int32, device=DEV)
    kw = dict(norm="layernorm", norm_eps=1e-5, norm_gamma=fff_lib.from_numpy(gamma, DEV),
              norm_beta=fff_lib.from_numpy(beta, DEV), out="residual", nodes_out=nodes)
    assert fff_lib.describe(x, wi, wo, 11, 1, mode="tiled", **kw).startswith("tiled<")
    y = fff_lib.forward(x, wi, wo, 11, 1, mode="tiled", y_dtype=TORCH_DT[yd], **kw)
    torch.cuda.synchronize()
    ref = oracle.block(L["x"], L["w_in"], L["w_out"], 11, 1, norm={"gamma": gamma, "beta": beta, "eps": 1e-5})
    fff_only = dict(ref, y=ref["fff"])
    rep = parity.assert_parity(ref["u"], L["w_in"], L["w_out"], 11, 1, fff_only, fff_lib.to_numpy(y),
                               nodes.cpu().numpy(), tol=tol_for("bf16", yd), base_dev=L["x"])
    flush_print(f"[gpu] tiled + LayerNorm y={yd}: {parity.summary(rep)}")


@pytest.mark.parametrize("name", ["4x9_h768_b16384_f32", "4x8_h768_b16384_f32"])
def test_tiled_multi_tree_full_size(fff_lib, name):
    """UltraFastBERT-4x9 and 4x8 at 16384 tokens through the leaf-tiled path: one tile pass per tree,
    in tree order, each adding to the running sum of the trees before it."""
    w = WORKLOADS[name]
    L = synth.make_layer(w.seed, w.n_tokens, w.hidden, w.depth, w.n_trees, w.x_dtype, w.w_dtype)
    check_layer(fff_lib, f"tiled {name}", L, w.depth, w.n_trees, w.y_dtype, mode="tiled")


@pytest.mark.parametrize("T,D,B,xd,wd,yd", [(2, 11, 9000, "bf16", "bf16", "bf16"), (3, 7, 2500, "f32", "bf16", "f32"),
                                          (16, 5, 3000, "bf16", "bf16", "f32"), (5, 6, 777, "f32", "f32", "bf16"),
                                          (2, 9, 1, "bf16", "bf16", "bf16")])
def test_tiled_multi_tree_shapes(fff_lib, T, D, B, xd, wd, yd):
    """Several trees, both weight types, bf16 outputs (the running sum then lives in the workspace),
    ragged and single-token batches."""
    L = layer(250 + T + D, B, 768, D, T, xd, wd)
    check_layer(fff_lib, f"tiled {T}x{D} B={B} {xd}/{wd}/{yd}", L, D, T, yd, mode="tiled")


@pytest.mark.parametrize("out", ["residual", "accumulate"])
@pytest.mark.parametrize("xd,yd", [("f32", "f32"), ("bf16", "bf16")])
def test_tiled_multi_tree_output_modes(fff_lib, out, xd, yd):
    B, T, D = 3000, 3, 9
    L = layer(260, B, 768, D, T, xd, "bf16")
    y0 = synth.make_x(261, B, 768, yd)
    got = run_fff(fff_lib, L, D, T, yd, mode="tiled", out=out, y_init=y0 if out == "accumulate" else None)
    ref = oracle.forward(L["x"], L["w_in"], L["w_out"], D, T)
    base = L["x"] if out == "residual" else y0
    rep = parity.assert_parity(L["x"], L["w_in"], L["w_out"], D, T, ref, got["y"], got["nodes"],
                               tol=tol_for("bf16", yd), base_dev=base)
    flush_print(f"[gpu] tiled {T}x{D} {out} {xd}/{yd}: {parity.summary(rep)}")


def test_tiled_multi_tree_spills_deterministic(fff_lib):
    """Clustered tokens overflow the buckets of every tree; two runs give the same bits."""
    B, T, D = 12000, 2, 10
    x = synth.make_clustered_x(270, B, 768, "bf16", n_centres=6)
    wi, wo = synth.make_weights(270, 768, D, T, "bf16")
    L = {"x": x, "w_in": wi, "w_out": wo}
    check_layer(fff_lib, "tiled 2x10 clustered", L, D, T, "f32", mode="tiled")
    a = run_fff(fff_lib, L, D, T, "f32", mode="tiled")
    b = run_fff(fff_lib, L, D, T, "f32", mode="tiled")
    assert np.array_equal(a["y"], b["y"]) and np.array_equal(a["nodes"], b["nodes"])


def test_tiled_leaf_pairs_plan(fff_lib):
    """Fewer than 16 tokens per leaf on average take a tile workgroup per pair of sibling leaves
    (depth <= 14); fuller leaves one per leaf."""
    def pairs(B, D, wd, T=1):
        x = torch.zeros(B, 768, dtype=torch.float32, device=DEV)
        w = torch.zeros(T, (2 << D) - 1, 768, dtype=TORCH_DT[wd], device=DEV)
        s = fff_lib.describe(x, w, w, D, T, mode="tiled")
        assert s.startswith("tiled<")
        return int(s.split("leaf_pairs=")[1].split()[0])
    assert pairs(16384, 11, "f32") == 1  # the paper's Table 2 shape: 8 tokens per leaf
    assert pairs(32767, 11, "f32") == 1 and pairs(32768, 11, "f32") == 0
    assert pairs(16384, 11, "bf16") == 1 and pairs(65536, 11, "bf16") == 0  # the headline: 32 per leaf
    assert pairs(3000, 14, "f32") == 1 and pairs(3000, 15, "f32") == 0  # two more rows fit 16 levels
    assert pairs(4096, 9, "f32", T=4) == 1 and pairs(16384, 9, "f32", T=4) == 0


@pytest.mark.parametrize("B,D,xd,yd", [(1, 11, "f32", "f32"), (7, 11, "f32", "bf16"), (100, 11, "bf16", "f32"),
                                       (2049, 5, "f32", "f32"), (5000, 14, "f32", "f32"), (16384, 11, "f32", "f32")])
def test_tiled_leaf_pairs(fff_lib, B, D, xd, yd):
    """Leaf pairs against the oracle: empty and single siblings (1 to 100 tokens), depth 5 (the
    fewest leaves), depth 14 (the two virtual rows fill the fourth step), the Table 2 shape."""
    L = layer(280 + B + D, B, 768, D, 1, xd, "f32")
    check_layer(fff_lib, f"tiled pairs B={B} D={D} {xd}/{yd}", L, D, 1, yd, mode="tiled")


def test_tiled_leaf_pairs_spills_deterministic(fff_lib):
    """Clustered tokens overflow some leaves: the pair of an overflowing leaf takes the per-token
    emit for both siblings; two runs give the same bits."""
    B, D = 20000, 11
    x = synth.make_clustered_x(290, B, 768, "f32", n_centres=8)
    wi, wo = synth.make_weights(290, 768, D, 1, "f32")
    L = {"x": x, "w_in": wi, "w_out": wo}
    assert "leaf_pairs=1" in fff_lib.describe(fff_lib.from_numpy(x, DEV), fff_lib.from_numpy(wi, DEV),
                                              fff_lib.from_numpy(wo, DEV), D, 1, mode="tiled")
    check_layer(fff_lib, "tiled pairs clustered", L, D, 1, "f32", mode="tiled")
    a = run_fff(fff_lib, L, D, 1, "f32", mode="tiled")
    b = run_fff(fff_lib, L, D, 1, "f32", mode="tiled")
    assert np.array_equal(a["y"], b["y"]) and np.array_equal(a["nodes"], b["nodes"])


def test_tiled_unsupported_shapes(fff_lib):
    L = layer(240, 64, 768, 4, 1, "f32", "f32")  # depth below 5
    with pytest.raises(fff_lib.FffError):
        run_fff(fff_lib, L, 4, 1, "f32", mode="tiled")
    L = layer(241, 64, 768, 5, 17, "f32", "f32")  # more than 16 trees
    with pytest.raises(fff_lib.FffError):
        run_fff(fff_lib, L, 5, 17, "f32", mode="tiled")
    L = layer(242, 64, 768, 16, 1, "bf16", "bf16")  # depth above 15
    with pytest.raises(fff_lib.FffError):
        run_fff(fff_lib, L, 16, 1, "bf16", mode="tiled")


# ----------------------------------------------------- MASKED (dense products)


@pytest.mark.parametrize("yd", ["bf16", "f32"])
@pytest.mark.parametrize("k,d,B", [(3072, 0, 131), (1536, 1, 64), (512, 2, 131), (64, 5, 257), (16, 7, 100),
                                   (1, 3, 5), (3, 4, 50), (200, 5, 33)])
def test_masked_shapes(fff_lib, k, d, B, yd):
    """The masked mode (logit GEMM, walk over the logits, output GEMM on split activations) against
    the oracle for shallow KxD shapes, ragged batches and both output types."""
    L = layer(400 + d + k, B, 768, d, k, "bf16", "bf16")
    check_layer(fff_lib, f"masked {k}x{d} B={B} y={yd}", L, d, k, yd, mode="masked")


@pytest.mark.parametrize("k,d,B", [(3072, 0, 67), (512, 2, 131), (64, 5, 257), (16, 7, 100), (1, 3, 5), (3, 4, 50),
                                   (200, 5, 33)])
def test_masked_f32_shapes(fff_lib, k, d, B):
    """fp32 x, W and y: both products are fp32 GEMMs and the activations go in whole.  N_T = 15 and
    93 take padded rows; 200 trees of depth 5 (N_T = 12600) the selection for rows wider than LDS."""
    L = layer(440 + d + k, B, 768, d, k, "f32", "f32")
    check_layer(fff_lib, f"masked f32 {k}x{d} B={B}", L, d, k, "f32", mode="masked")


@pytest.mark.parametrize("dt,H", [("bf16", 200), ("bf16", 8), ("f32", 104), ("f32", 8)])
def test_masked_ragged_hidden(fff_lib, dt, H):
    """A hidden size that is not a whole number of the products' K steps (64 bf16 or 32 fp32
    elements) takes the register-staged product kernel, which masks the K tail."""
    L = layer(460 + H, 300, H, 2, 16, dt, dt)
    check_layer(fff_lib, f"masked {dt} H={H}", L, 2, 16, dt, mode="masked")


@pytest.mark.parametrize("out", ["residual", "accumulate"])
def test_masked_f32_output_modes(fff_lib, out):
    L = layer(450, 300, 768, 2, 16, "f32", "f32")
    y0 = synth.make_x(451, 300, 768, "f32")
    got = run_fff(fff_lib, L, 2, 16, "f32", mode="masked", out=out, y_init=y0 if out == "accumulate" else None)
    ref = oracle.forward(L["x"], L["w_in"], L["w_out"], 2, 16)
    base = L["x"] if out == "residual" else y0
    parity.assert_parity(L["x"], L["w_in"], L["w_out"], 2, 16, ref, got["y"], got["nodes"], tol=1e-5,
                         base_dev=base)


@pytest.mark.parametrize("dt,out", [("f32", "residual"), ("f32", "accumulate"), ("bf16", "residual"),
                                    ("bf16", "accumulate"), ("bf16", "store")])
def test_masked_split_output_modes(fff_lib, dt, out):
    """At 300 tokens the output product (K = N_T' fp32 or 2 N_T' bf16 columns) is split along K;
    the reduction applies the layer's output form (residual, accumulate, plain store)."""
    k, d, B = 256, 3, 300
    L = layer(470 + len(out), B, 768, d, k, dt, dt)
    y0 = synth.make_x(471, B, 768, dt) if out == "accumulate" else None
    got = run_fff(fff_lib, L, d, k, dt, mode="masked", out=out, y_init=y0)
    ref = oracle.forward(L["x"], L["w_in"], L["w_out"], d, k)
    base = None if out == "store" else (L["x"] if out == "residual" else y0)
    parity.assert_parity(L["x"], L["w_in"], L["w_out"], d, k, ref, got["y"], got["nodes"],
                         tol=1e-5 if dt == "f32" else 2e-2, base_dev=base)


@pytest.mark.parametrize("out", ["residual", "accumulate"])
def test_masked_output_modes(fff_lib, out):
    L = layer(420, 1000, 768, 3, 32, "bf16", "bf16")
    y0 = synth.make_x(421, 1000, 768, "bf16")
    got = run_fff(fff_lib, L, 3, 32, "bf16", mode="masked", out=out, y_init=y0 if out == "accumulate" else None)
    ref = oracle.forward(L["x"], L["w_in"], L["w_out"], 3, 32)
    base = L["x"] if out == "residual" else y0
    parity.assert_parity(L["x"], L["w_in"], L["w_out"], 3, 32, ref, got["y"], got["nodes"], tol=2e-2,
                         base_dev=base)


@pytest.mark.parametrize("k,B,dt,yd,out,act", [(3072, 131, "bf16", "bf16", "store", "gelu"),
                                                (3072, 131, "bf16", "f32", "accumulate", "gelu_tanh"),
                                                (3072, 67, "f32", "f32", "accumulate", "gelu"),
                                                (100, 1000, "bf16", "bf16", "residual", "identity"),
                                                (100, 1000, "f32", "f32", "store", "gelu"),
                                                (3072, 37, "bf16", "bf16", "accumulate", "gelu"),
                                                (3072, 64, "f32", "f32", "residual", "gelu_tanh"),
                                                (3, 5, "bf16", "bf16", "store", "gelu")])
def test_masked_depth0_without_records(fff_lib, k, B, dt, yd, out, act):
    """Depth 0 with no records: the logit product stores the activations (two bf16 parts, or
    whole for fp32) over the padded rows itself, with no selection pass (bf16 operands with an
    fp32 output, three parts, keep the selection).  Against the oracle (at depth 0 every path is
    the root, so the paths are the oracle's), and bit for bit against the same call with records,
    which selects from stored logits.  k = 100 pads the rows from 100 to 128 columns and k = 3
    from 3 to 64; 37 and 64 tokens split the logit product along K."""
    L = layer(480 + k + B, B, 768, 0, k, dt, dt)
    y0 = synth.make_x(481, B, 768, yd) if out == "accumulate" else None
    flush_print(f"[gpu] masked depth 0 without records: k={k} B={B} {dt} y={yd} {out} {act}")
    got = run_fff(fff_lib, L, 0, k, yd, record=False, y_init=y0, mode="masked", out=out, act=act)
    rec = run_fff(fff_lib, L, 0, k, yd, y_init=y0, mode="masked", out=out, act=act)
    ref = oracle.forward(L["x"], L["w_in"], L["w_out"], 0, k, act=act)
    base = None if out == "store" else (L["x"] if out == "residual" else y0)
    parity.assert_parity(L["x"], L["w_in"], L["w_out"], 0, k, ref, got["y"], ref["nodes"], tol=tol_for(dt, yd),
                         act=act, base_dev=base)
    assert np.array_equal(got["y"].view(np.uint8), rec["y"].view(np.uint8))


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_masked_depth0_full_size_sampled(fff_lib, dt):
    """3072 trees of depth 0 at 16384 tokens, as the KxD sweep times it: AUTO (masked, the logit
    product storing the activations), no records; 384 sampled tokens against the oracle."""
    B, k = 16384, 3072
    L = layer(490, B, 768, 0, k, dt, dt)
    x = fff_lib.from_numpy(L["x"], DEV)
    wi = fff_lib.from_numpy(L["w_in"], DEV)
    wo = fff_lib.from_numpy(L["w_out"], DEV)
    y = torch.full((B, 768), float("nan"), dtype=TORCH_DT[dt], device=DEV)
    assert fff_lib.describe(x, wi, wo, 0, k, y).startswith("masked<")
    flush_print(f"[gpu] masked depth 0 full size: k={k} B={B} {dt}")
    fff_lib.forward(x, wi, wo, 0, k, y)
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(491).choice(B, 384, replace=False))
    ref = oracle.forward(L["x"][rows], L["w_in"], L["w_out"], 0, k)
    parity.assert_parity(L["x"], L["w_in"], L["w_out"], 0, k, ref, fff_lib.to_numpy(y), rows=rows,
                         tol=tol_for(dt, dt))


def test_masked_mode_limits_and_auto(fff_lib):
    """Masked needs bf16 x and W, or fp32 x, W and y, and depth <= 7; AUTO takes it at depth <= 5
    for 16 bf16 trees or more, or 12 and 16384 tokens, and at depth <= 4 for 32 fp32 trees or more
    (planning only)."""
    L = layer(430, 64, 768, 3, 8, "f32", "bf16")
    x, wi, wo = (fff_lib.from_numpy(L[k], DEV) for k in ("x", "w_in", "w_out"))
    with pytest.raises(fff_lib.FffError):
        fff_lib.forward(x, wi, wo, 3, 8, mode="masked")  # fp32 x, bf16 W
    L = layer(431, 64, 768, 3, 8, "f32", "f32")
    x, wi, wo = (fff_lib.from_numpy(L[k], DEV) for k in ("x", "w_in", "w_out"))
    with pytest.raises(fff_lib.FffError):
        fff_lib.forward(x, wi, wo, 3, 8, torch.empty((64, 768), dtype=torch.bfloat16, device=DEV),
                        mode="masked")  # fp32 x and W, bf16 y
    w8 = torch.zeros((1, (1 << 9) - 1, 768), dtype=torch.bfloat16, device=DEV)
    xb = torch.zeros((16384, 768), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(fff_lib.FffError):
        fff_lib.forward(xb[:64], w8, w8, 8, 1, mode="masked")  # depth 8
    w16 = torch.zeros((16, 15, 768), dtype=torch.bfloat16, device=DEV)
    assert fff_lib.describe(xb[:512], w16, w16, 3, 16).startswith("masked<")  # 16 trees
    w12 = torch.zeros((12, 15, 768), dtype=torch.bfloat16, device=DEV)
    assert fff_lib.describe(xb, w12, w12, 3, 12).startswith("masked<")  # 12 trees, 16384 tokens
    assert not fff_lib.describe(xb[:8192], w12, w12, 3, 12).startswith("masked<")  # 12 trees, 8192 tokens
    w8t = torch.zeros((8, 15, 768), dtype=torch.bfloat16, device=DEV)
    assert not fff_lib.describe(xb, w8t, w8t, 3, 8).startswith("masked<")  # 8 trees: the walk
    w1 = torch.zeros((1, 15, 768), dtype=torch.bfloat16, device=DEV)
    assert fff_lib.describe(xb, w1, w1, 3, 1).startswith("descent<")  # one tree: the walk
    w6 = torch.zeros((16, 127, 768), dtype=torch.bfloat16, device=DEV)
    assert not fff_lib.describe(xb[:4096], w6, w6, 6, 16).startswith("masked<")  # depth 6: the walk
    xf = torch.zeros((4096, 768), dtype=torch.float32, device=DEV)
    w4 = torch.zeros((32, 31, 768), dtype=torch.float32, device=DEV)
    assert fff_lib.describe(xf, w4, w4, 4, 32).startswith("masked<fp32")  # fp32, depth 4, 32 trees
    assert not fff_lib.describe(xf, w4[:16], w4[:16], 4, 16).startswith("masked<")  # 16 fp32 trees: the walk
    w5 = torch.zeros((32, 63, 768), dtype=torch.float32, device=DEV)
    assert not fff_lib.describe(xf, w5, w5, 5, 32).startswith("masked<")  # fp32, depth 5: the walk


@pytest.mark.parametrize("dt,B,d", [("bf16", 1024, 5), ("bf16", 4096, 7), ("f32", 1024, 4)])
def test_auto_eight_trees_grouped_parity(fff_lib, dt, B, d):
    """What AUTO plans for eight trees at small batches (GROUPED, its walk one tree per XCD) against
    the oracle."""
    L = layer(490 + d, B, 768, d, 8, dt, dt)
    x = fff_lib.from_numpy(L["x"], DEV)
    wi = fff_lib.from_numpy(L["w_in"], DEV)
    assert fff_lib.describe(x, wi, wi, d, 8).startswith("grouped<")
    check_layer(fff_lib, f"auto 8 trees {dt} B={B} d={d}", L, d, 8, dt)


def test_binding_workspace_per_stream(fff_lib):
    """The binding's cached workspace is one per (device, stream): two tiled forwards enqueued on two
    streams at once, each on its own inputs, both match the oracle, on different buffers."""
    d, B = 9, 8192
    Ls = [layer(480 + i, B, 768, d, 1, "bf16", "bf16") for i in range(2)]
    dev_in = [[fff_lib.from_numpy(L[k], DEV) for k in ("x", "w_in", "w_out")] for L in Ls]
    ys = [torch.empty((B, 768), dtype=torch.bfloat16, device=DEV) for _ in Ls]
    recs = [torch.empty((B, 1, d + 1), dtype=torch.int32, device=DEV) for _ in Ls]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    main = torch.cuda.current_stream()
    for s in streams:
        s.wait_stream(main)
    for i, s in enumerate(streams):
        with torch.cuda.stream(s):
            x, wi, wo = dev_in[i]
            fff_lib.forward(x, wi, wo, d, 1, ys[i], mode="tiled", nodes_out=recs[i])
    torch.cuda.synchronize()
    w = [fff_lib.fff.workspace_for(B, d, 1, 768, DEV, s).data_ptr() for s in streams]
    assert w[0] != w[1]
    for i, L in enumerate(Ls):
        ref = oracle.forward(L["x"], L["w_in"], L["w_out"], d, 1)
        parity.assert_parity(L["x"], L["w_in"], L["w_out"], d, 1, ref, fff_lib.to_numpy(ys[i]),
                             recs[i].cpu().numpy(), tol=2e-2)


def test_auto_multi_tree_deep_plans(fff_lib):
    """2, 4 or 8 trees of depth >= 7 plan the tree-affine walk: leaf-tiled with fp32 weights at
    depth >= 11 from 8 tokens per leaf or at depth >= 9 from 32 per leaf;
    otherwise GROUPED at large batches; the fused kernel below (planning only)."""
    def plan(T, d, B, dt):
        t = torch.bfloat16 if dt == "bf16" else torch.float32
        x = torch.zeros((B, 768), dtype=t, device=DEV)
        w = torch.zeros((T, (1 << (d + 1)) - 1, 768), dtype=t, device=DEV)
        return fff_lib.describe(x, w, w, d, T).split("<")[0]
    assert plan(4, 9, 16384, "f32") == "tiled"      # UltraFastBERT-4x9: 32 per leaf
    assert plan(4, 9, 8192, "f32") == "descent"     # 16 per leaf
    assert plan(4, 10, 16384, "f32") == "tiled"     # 16 per leaf at depth 10
    assert plan(4, 10, 8192, "f32") == "descent"
    assert plan(4, 8, 16384, "f32") == "descent"    # depth 8
    assert plan(8, 11, 65536, "f32") == "tiled"
    assert plan(2, 11, 16384, "f32") == "tiled"     # 8 per leaf at depth 11
    assert plan(2, 9, 65536, "f32") == "tiled"      # 128 per leaf
    assert plan(2, 8, 65536, "f32") == "grouped"    # depth 8
    assert plan(8, 8, 16384, "f32") == "grouped"
    assert plan(4, 7, 16384, "f32") == "descent"
    assert plan(4, 9, 4096, "bf16") == "grouped"
    assert plan(4, 7, 16384, "bf16") == "descent"   # depth 7: from 65536 tokens
    assert plan(2, 9, 16384, "bf16") == "descent"
    assert plan(2, 9, 65536, "bf16") == "grouped"
    assert plan(8, 7, 65536, "bf16") == "grouped"
    assert plan(4, 6, 65536, "bf16") == "descent"   # depth 6


@pytest.mark.parametrize("T,d,B,dt,want", [(4, 9, 4096, "bf16", "grouped<"), (8, 8, 16384, "f32", "grouped<"),
                                           (2, 11, 16384, "f32", "tiled<")])
def test_auto_multi_tree_deep_parity(fff_lib, T, d, B, dt, want):
    """The plans AUTO takes for deep multi-tree layers against the oracle."""
    L = layer(520 + T + d, B, 768, d, T, dt, dt)
    x = fff_lib.from_numpy(L["x"], DEV)
    wi = fff_lib.from_numpy(L["w_in"], DEV)
    assert fff_lib.describe(x, wi, wi, d, T).startswith(want)
    check_layer(fff_lib, f"auto {T} trees {dt} B={B} d={d}", L, d, T, dt)


def test_auto_eight_trees_small_batches(fff_lib):
    """Eight trees at small batches plan GROUPED (its walk one tree per XCD), larger batches the
    fused DESCENT kernel (planning only)."""
    for wd, small, large in (("bf16", 2048, 4096), ("f32", 1024, 2048)):
        dt = torch.bfloat16 if wd == "bf16" else torch.float32
        w = torch.zeros((8, 31, 768), dtype=dt, device=DEV)
        for B, want in ((small, "grouped<"), (large, "descent<")):
            x = torch.zeros((B, 768), dtype=dt, device=DEV)
            assert fff_lib.describe(x, w, w, 4, 8).startswith(want), (wd, B)
    w7 = torch.zeros((8, 255, 768), dtype=torch.bfloat16, device=DEV)
    x = torch.zeros((4096, 768), dtype=torch.bfloat16, device=DEV)
    assert fff_lib.describe(x, w7, w7, 7, 8).startswith("grouped<")  # depth 7: up to 4096 tokens
    assert fff_lib.describe(x[:16], w7[:4], w7[:4], 7, 4).startswith(("descent<", "subtree<"))  # four trees


# ----------------------------------------------------- SUBTREE (a workgroup per token)


@pytest.mark.parametrize("H,d,k,B,xd,wd,yd", [
    (768, 11, 1, 5, "bf16", "bf16", "bf16"),     # 16-lane dots, 6 levels per step: 2 steps
    (768, 0, 1, 3, "bf16", "bf16", "f32"),       # one level
    (768, 3, 2, 7, "f32", "bf16", "f32"),        # one partial step, two trees
    (768, 12, 1, 4, "bf16", "f32", "bf16"),      # 32-lane dots, 5 levels per step
    (1024, 9, 3, 6, "f32", "f32", "f32"),
    (1024, 10, 1, 9, "f32", "bf16", "f32"),      # 512-thread workgroups, 5 levels per step
    (4096, 13, 1, 3, "bf16", "bf16", "bf16"),    # 64-lane dots, 4 levels per step (last step 2)
    (4096, 7, 1, 2, "f32", "bf16", "f32"),       # 512-thread workgroups, 3 levels per step
    (4096, 6, 2, 2, "f32", "f32", "f32"),
])
def test_subtree_shapes(fff_lib, H, d, k, B, xd, wd, yd):
    """SUBTREE mode (whole subtrees of logits per step) against the oracle, with the records."""
    L = layer(500 + H + d + k, B, H, d, k, xd, wd)
    check_layer(fff_lib, f"subtree H={H} {k}x{d} B={B} {xd}/{wd}/{yd}", L, d, k, yd, mode="subtree")


def test_subtree_many_tokens(fff_lib):
    """More tokens than workgroups: each workgroup loops over tokens."""
    L = layer(530, 1500, 768, 4, 1, "bf16", "bf16")
    check_layer(fff_lib, "subtree B=1500", L, 4, 1, "bf16", mode="subtree")


@pytest.mark.parametrize("out", ["residual", "accumulate"])
@pytest.mark.parametrize("xd,wd", [("bf16", "bf16"), ("f32", "f32")])
def test_subtree_output_modes(fff_lib, out, xd, wd):
    """y = x + FFF(x) and y += FFF(x).  A bf16 y holds the rounding of the whole sum, whose error
    scales with the base, not with FFF(x): there every element must lie within one bf16 spacing of
    the fp64 total plus the fp32 bar on FFF(x)."""
    B = 33
    L = layer(540, B, 768, 9, 2, xd, wd)
    y0 = synth.make_x(541, B, 768, xd)
    got = run_fff(fff_lib, L, 9, 2, xd, mode="subtree", out=out, y_init=y0 if out == "accumulate" else None)
    ref = oracle.forward(L["x"], L["w_in"], L["w_out"], 9, 2)
    base = L["x"] if out == "residual" else y0
    parity.assert_parity(L["x"], L["w_in"], L["w_out"], 9, 2, ref, got["y"], got["nodes"],
                         tol=2e-2 if xd == "bf16" else 1e-5, base_dev=base)


def test_subtree_auto_and_limits(fff_lib):
    """AUTO takes SUBTREE for at most 4 trees of depth >= 5 and 256 token-tree pairs (32 at hidden
    4096, 128 with fp32 weights from depth 11); no LayerNorm, no other widths."""
    xb = torch.zeros((300, 768), dtype=torch.bfloat16, device=DEV)
    w11 = torch.zeros((1, (1 << 12) - 1, 768), dtype=torch.bfloat16, device=DEV)
    assert fff_lib.describe(xb[:256], w11, w11, 11, 1).startswith("subtree<")
    assert fff_lib.describe(xb[:1], w11, w11, 11, 1).startswith("subtree<")
    assert not fff_lib.describe(xb[:257], w11, w11, 11, 1).startswith("subtree<")
    w5 = torch.zeros((4, 63, 768), dtype=torch.bfloat16, device=DEV)
    assert fff_lib.describe(xb[:64], w5, w5, 5, 4).startswith("subtree<")  # 4 trees x 64 tokens
    assert not fff_lib.describe(xb[:65], w5, w5, 5, 4).startswith("subtree<")
    w4 = torch.zeros((1, 31, 768), dtype=torch.bfloat16, device=DEV)
    assert not fff_lib.describe(xb[:8], w4, w4, 4, 1).startswith("subtree<")  # depth 4
    w5t = torch.zeros((5, 63, 768), dtype=torch.bfloat16, device=DEV)
    assert not fff_lib.describe(xb[:8], w5t, w5t, 5, 5).startswith("subtree<")  # 5 trees
    x4 = torch.zeros((40, 4096), dtype=torch.bfloat16, device=DEV)
    w12 = torch.zeros((1, (1 << 13) - 1, 4096), dtype=torch.bfloat16, device=DEV)
    assert fff_lib.describe(x4[:32], w12, w12, 12, 1).startswith("subtree<")
    assert not fff_lib.describe(x4[:33], w12, w12, 12, 1).startswith("subtree<")
    # fp32 weights from depth 11: 128 pairs
    xf = torch.zeros((300, 768), dtype=torch.float32, device=DEV)
    wf11 = torch.zeros((1, (1 << 12) - 1, 768), dtype=torch.float32, device=DEV)
    assert fff_lib.describe(xf[:128], wf11, wf11, 11, 1).startswith("subtree<")
    assert fff_lib.describe(xf[:129], wf11, wf11, 11, 1).startswith("descent<")
    wf9 = torch.zeros((1, (1 << 10) - 1, 768), dtype=torch.float32, device=DEV)
    assert fff_lib.describe(xf[:256], wf9, wf9, 9, 1).startswith("subtree<")
    x5 = torch.zeros((4, 640), dtype=torch.bfloat16, device=DEV)
    w5w = torch.zeros((1, 63, 640), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(fff_lib.FffError):
        fff_lib.forward(x5, w5w, w5w, 5, 1, mode="subtree")  # no kernel for hidden 640


_MASKED_CHILD = r"""
import hashlib, sys
import torch
sys.path.insert(0, sys.argv[1])
import paper_2311_10770_amd as fff
from paper_2311_10770_amd import synth
fff.load_library()
dev = torch.device("cuda:0")
out = []
for xd, yd, k, d, B in (("bf16", "bf16", 512, 2, 4096), ("bf16", "f32", 64, 5, 4096), ("f32", "f32", 128, 4, 4096),
                        ("bf16", "bf16", 3072, 0, 256), ("f32", "f32", 256, 3, 300)):
    L = synth.make_layer(77, B, 768, d, k, xd, xd)
    x, wi, wo = (fff.from_numpy(L[n], dev) for n in ("x", "w_in", "w_out"))
    y = torch.empty((B, 768), dtype=torch.bfloat16 if yd == "bf16" else torch.float32, device=dev)
    fff.forward(x, wi, wo, d, k, y, mode="masked")
    torch.cuda.synchronize()
    out.append(hashlib.sha256(y.view(torch.uint8).cpu().numpy().tobytes()).hexdigest())
print(" ".join(out))
"""


def test_masked_bits_do_not_depend_on_the_process():
    """Masked mode's products run a fixed algorithm per shape (no timing-based choice; a K split and
    its reduction order fixed by the shapes and the CU count: the 256- and 300-token cases split the
    output product), so two fresh processes produce the same output bits."""
    import subprocess
    import sys

    from tests.conftest import ROOT

    runs = []
    for i in range(2):
        flush_print(f"[gpu] masked bits, fresh process {i}")
        r = subprocess.run([sys.executable, "-c", _MASKED_CHILD, str(ROOT)], capture_output=True, text=True,
                           timeout=300)
        assert r.returncode == 0, r.stderr[-2000:]
        runs.append(r.stdout.strip().splitlines()[-1])
    assert runs[0] == runs[1], runs
