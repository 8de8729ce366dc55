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


def _fp32_forward(x, w_in, w_out, depth, parts=0):
    """An honest fp32 evaluation of one tree, vectorised over tokens (numpy float32 dot products,
    activations rounded once to fp32, fp32 accumulation).  ``parts`` > 0: each activation replaced
    by the sum of its first ``parts`` bf16 parts, as a split-activation emit would use it."""
    x32 = parity.widen(x).astype(np.float32)
    wi = parity.widen(w_in[0]).astype(np.float32)
    wo = parity.widen(w_out[0]).astype(np.float32)
    B = x32.shape[0]
    n = np.zeros(B, dtype=np.int64)
    y = np.zeros_like(x32)
    for level in range(depth + 1):
        l = np.einsum("bh,bh->b", x32, wi[n])
        a = parity.act_values(l.astype(np.float64), "gelu").astype(np.float32)
        if parts:
            rest, used = a.copy(), np.zeros_like(a)
            for _ in range(parts):
                p = parity.widen(oracle.round_bf16(rest.astype(np.float64))).astype(np.float32)
                used += p
                rest = rest - p
            a = used
        y += a[:, None] * wo[n]
        if level < depth:
            n = 2 * n + 1 + (l > 0)
    return y


def test_honest_fp32_meets_the_raw_bar_without_exceptions():
    """The depth-11, hidden-768 shape of the paper's speed test evaluated in plain fp32 meets the raw
    1e-5 bar on every token, ill-conditioned or not: no allowance is used."""
    L = synth.make_layer(2, 600, 768, 11, 1, "f32", "f32")
    ref = oracle.forward(L["x"], L["w_in"], L["w_out"], 11, 1)
    y = _fp32_forward(L["x"], L["w_in"], L["w_out"], 11)
    rep = parity.check(L["x"], L["w_in"], L["w_out"], 11, 1, ref, y, ref["nodes"])
    assert rep["ok"], parity.summary(rep)
    assert rep["n_conditioned"] == 0 and rep["max_normwise_err_raw"] < 1e-5


def test_well_conditioned_token_gets_no_allowance(case):
    """An error of 3e-5 relative fails on a typical token, however large ||x|| ||W|| is."""
    L, ref = case
    y = ref["y"].copy()
    y[9] += 3e-5 * np.linalg.norm(ref["y"][9]) * np.eye(1, y.shape[1], 4)[0]
    rep = parity.check(L["x"], L["w_in"], L["w_out"], 6, 2, ref, y, ref["nodes"])
    assert not rep["ok"] and rep["value_failures"][0][0] == 9 and rep["n_conditioned"] == 0


def _depth0_token(logit):
    """One node of hidden 768 and a typical token whose logit is set to ``logit``."""
    H = 768
    rng = np.random.default_rng(8)
    w_in = (rng.standard_normal((1, 1, H)) / np.sqrt(H)).astype(np.float32)
    w_out = (rng.standard_normal((1, 1, H)) / np.sqrt(H)).astype(np.float32)
    w = w_in[0, 0].astype(np.float64)
    r = rng.standard_normal(H)
    r -= (r @ w) / (w @ w) * w                # a typical token, orthogonal to the row ...
    x = (r + logit * w / (w @ w))[None].astype(np.float32)  # ... plus a component giving the logit
    return x, w_in, w_out


def test_ill_conditioned_class_and_its_allowance():
    """Depth 0 with a logit of 1e-4: y = act(l) W_out[0] and l is a sum of products some 10^5 times
    larger than itself, so kappa is far above KAPPA_MAX.  A logit off by 4 fp32 roundings of those
    magnitudes is accepted -- counted, and only when the caller allows it; 1000 times that is not
    rounding.  At a logit of -2 the token is well conditioned and a 3e-5 error fails."""
    x, w_in, w_out = _depth0_token(1e-4)
    ref = oracle.forward(x, w_in, w_out, 0, 1)
    l = ref["logits"][0, 0, 0]
    slope = parity.act_slope(np.array([l]), "gelu")[0]
    S = float(np.abs(x[0].astype(np.float64) * w_in[0, 0]).sum())
    dl = 4 * 2.0 ** -24 * S
    y_dev = ref["y"] + slope * dl * w_out[0, 0]
    rep = parity.check(x, w_in, w_out, 0, 1, ref, y_dev, ref["nodes"], max_conditioned=1)
    assert rep["ok"] and rep["n_ill_conditioned"] == 1 and rep["n_conditioned"] == 1, parity.summary(rep)
    assert rep["max_normwise_err_raw"] > 1e-5 and rep["max_kappa"] > parity.KAPPA_MAX
    assert not parity.check(x, w_in, w_out, 0, 1, ref, y_dev, ref["nodes"])["ok"]  # max_conditioned = 0
    y_bad = ref["y"] + slope * 1000 * dl * w_out[0, 0]
    assert not parity.check(x, w_in, w_out, 0, 1, ref, y_bad, ref["nodes"], max_conditioned=1)["ok"]
    x, w_in, w_out = _depth0_token(-2.0)
    ref = oracle.forward(x, w_in, w_out, 0, 1)
    y_dev = ref["y"] * (1 + 3e-5)
    rep = parity.check(x, w_in, w_out, 0, 1, ref, y_dev, ref["nodes"], max_conditioned=1)
    assert not rep["ok"] and rep["n_ill_conditioned"] == 0


def test_kappa_matches_its_closed_form_at_depth_zero():
    """One node: y = act(l) W_out[0], so kappa = 1 + |act'(l)| S / |act(l)|, S = sum |x_i W_in_i|."""
    x, w_in, w_out = _depth0_token(-2.0)
    ref = oracle.forward(x, w_in, w_out, 0, 1)
    l = float(ref["logits"][0, 0, 0])
    a = parity.act_values(np.array(l), "gelu")
    s = parity.act_slope(np.array(l), "gelu")
    S = float(np.abs(x[0].astype(np.float64) * w_in[0, 0]).sum())
    kappa, _ = parity.conditioning(x, w_in, w_out, 0, 1, ref["nodes"], ref["logits"], ref["y"], "gelu")
    assert kappa[0] == pytest.approx(1 + s * S / abs(a), rel=1e-12)


def test_bf16_elementwise_bound_pins_the_activation_split():
    """bf16 outputs: an fp32 emit on hi + mid bf16 parts of each activation, rounded to bf16, passes
    the elementwise bound; hi alone (a dropped mid part) fails it, although it still meets the
    normwise 2e-2 bar."""
    L = synth.make_layer(3, 400, 768, 11, 1, "bf16", "bf16")
    ref = oracle.forward(L["x"], L["w_in"], L["w_out"], 11, 1)
    good = oracle.round_bf16(_fp32_forward(L["x"], L["w_in"], L["w_out"], 11, parts=2).astype(np.float64))
    rep = parity.check(L["x"], L["w_in"], L["w_out"], 11, 1, ref, good, ref["nodes"], tol=2e-2)
    assert rep["ok"] and rep["bf16_elem_excess"] <= 1.0, parity.summary(rep)
    bad = oracle.round_bf16(_fp32_forward(L["x"], L["w_in"], L["w_out"], 11, parts=1).astype(np.float64))
    rep = parity.check(L["x"], L["w_in"], L["w_out"], 11, 1, ref, bad, ref["nodes"], tol=2e-2)
    assert not rep["ok"] and rep["n_bf16_elem_failures"] > 0 and rep["n_value_failures"] == 0


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
