"""The GPU-vs-oracle acceptance checker itself, exercised on the CPU with planted differences."""
import numpy as np
import pytest

import oracle
from oracle import parity
from paper_2311_10770_amd import synth


@pytest.fixture(scope="module")
def case():
    L = synth.make_layer(5, 400, 64, 6, 2, "f32", "f32")
    ref = oracle.forward(L["x"], L["w_in"], L["w_out"], 6, 2)
    return L, ref


def test_exact_copy_passes(case):
    L, ref = case
    rep = parity.check(L["x"], L["w_in"], L["w_out"], 6, 2, ref, ref["y"].astype(np.float32), ref["nodes"])
    assert rep["ok"] and rep["n_path_divergent"] == 0


def test_small_value_error_passes_large_fails(case):
    L, ref = case
    y = ref["y"] * (1 + 2e-6)
    assert parity.check(L["x"], L["w_in"], L["w_out"], 6, 2, ref, y, ref["nodes"])["ok"]
    y = ref["y"].copy()
    y[17] *= 1 + 1e-3
    rep = parity.check(L["x"], L["w_in"], L["w_out"], 6, 2, ref, y, ref["nodes"])
    assert not rep["ok"] and rep["value_failures"][0][0] == 17


def test_branch_flip_off_tie_fails(case):
    L, ref = case
    nodes = ref["nodes"].copy()
    b, t = 3, 1
    nodes[b, t, 2] = nodes[b, t, 2] + (1 if nodes[b, t, 2] % 2 else -1)  # sibling
    for lvl in range(3, 7):
        nodes[b, t, lvl] = 2 * nodes[b, t, lvl - 1] + 1
    rep = parity.check(L["x"], L["w_in"], L["w_out"], 6, 2, ref, ref["y"], nodes)
    assert not rep["ok"] and rep["path_failures"][0][:2] == (3, 1)


def test_branch_flip_at_near_tie_is_accepted():
    H, D = 64, 4
    rng = np.random.default_rng(3)
    w_in = rng.standard_normal((1, 31, H)).astype(np.float32)
    w_out = rng.standard_normal((1, 31, H)).astype(np.float32)
    w0 = w_in[0, 0].astype(np.float64)
    x = rng.standard_normal((1, H))
    x[0] -= (x[0] @ w0) / (w0 @ w0) * w0
    x = x.astype(np.float32)
    ref = oracle.forward(x, w_in, w_out, D, 1)
    assert ref["near_tie"][0, 0, 0]
    other = 2 if ref["nodes"][0, 0, 1] == 1 else 1
    # walk the other subtree by signs, as a device that rounded the root logit the other way would
    path = [0, other]
    xd = x[0].astype(np.float64)
    for _ in range(2, D + 1):
        n = path[-1]
        path.append(2 * n + 1 + (1 if xd @ w_in[0, n].astype(np.float64) > 0 else 0))
    y_dev, _ = oracle.eval_path(x[0], w_in, w_out, D, 1, np.array([path]))
    rep = parity.check(x, w_in, w_out, D, 1, ref, y_dev[None], np.array([[path]], dtype=np.int32))
    assert rep["ok"] and rep["n_path_divergent"] == 1 and rep["n_near_tie"] == 1


def test_illegal_device_path_fails(case):
    L, ref = case
    nodes = ref["nodes"].copy()
    nodes[5, 0, 4] = 0
    rep = parity.check(L["x"], L["w_in"], L["w_out"], 6, 2, ref, ref["y"], nodes)
    assert not rep["ok"]


def test_conditioning_allowance_only_covers_logit_rounding():
    # one node, strongly negative logit: tiny y, large relative sensitivity
    H = 768
    rng = np.random.default_rng(8)
    w_in = (rng.standard_normal((1, 1, H)) / np.sqrt(H)).astype(np.float32)
    w_out = (rng.standard_normal((1, 1, H)) / np.sqrt(H)).astype(np.float32)
    w = w_in[0, 0].astype(np.float64)
    r = rng.standard_normal(H)
    r -= (r @ w) / (w @ w) * w                # a typical token, orthogonal to the row ...
    x = (r - 4.2 * w / (w @ w))[None].astype(np.float32)  # ... plus a component giving logit -4.2
    ref = oracle.forward(x, w_in, w_out, 0, 1)
    l = ref["logits"][0, 0, 0]
    assert l < -3
    slope = parity.act_slope(np.array([l]), "gelu")[0]
    # a logit off by 4 units of fp32 rounding of ||x|| ||w||
    dl = 4 * 2.0 ** -24 * np.linalg.norm(x) * np.linalg.norm(w_in[0])
    y_dev = ref["y"] + slope * dl * w_out[0, 0]
    rep = parity.check(x, w_in, w_out, 0, 1, ref, y_dev, ref["nodes"])
    assert rep["ok"] and rep["n_conditioned"] == 1 and rep["max_normwise_err_raw"] > 1e-5
    # 1000 units is not rounding
    y_bad = ref["y"] + slope * 250 * dl * w_out[0, 0]
    assert not parity.check(x, w_in, w_out, 0, 1, ref, y_bad, ref["nodes"])["ok"]


def test_bf16_total_excess_accepts_rounding_and_rejects_a_spacing_error():
    """The residual-output bound: rounding of x + f passes; an error of two spacings fails; tiny totals
    are judged against the FFF bar, not their own spacing."""
    from paper_2311_10770_amd import synth

    rng = np.random.default_rng(7)
    x = synth.as_dtype(rng.standard_normal((50, 64)).astype(np.float32), "bf16")
    f = rng.standard_normal((50, 64)) * 0.1
    total = parity.widen(x) + f
    stored = oracle.round_bf16(total)
    assert parity.bf16_total_excess(stored, total, f, 1e-5) <= 0.5 + 1e-9
    bad = stored.copy()
    bad[3, 5] = np.uint16(int(bad[3, 5]) + 2)  # two spacings off (same binade)
    assert parity.bf16_total_excess(bad, total, f, 1e-5) > 1.0
    # a total that cancels to ~1e-9: one bf16 spacing there is tiny, the FFF bar (1e-5 ||f||) is not
    t2 = total.copy()
    t2[0, 0] = 1e-9
    s2 = oracle.round_bf16(t2)
    s2[0, 0] = oracle.round_bf16(np.array([1e-9 + 1e-6]))[0]
    assert parity.bf16_total_excess(s2, t2, f, 1e-5) <= 1.0
