"""GPU-versus-oracle acceptance check -- TEST INFRASTRUCTURE ONLY.

Rules (paths first, then values):

1. Paths.  For every (token, tree) the device path is walked level by level.
   At the first level where its node differs from the oracle's, the oracle
   must have flagged the parent visit as a near tie
   (|logit| < tie_rel * ||x|| * ||W_in row||).  From there on the device path
   is re-evaluated in fp64 along its own nodes, and every later step must
   follow the sign of its fp64 logit (0 goes left) or be a near tie itself.
   Any other difference fails.
2. Counts.  ``n_near_tie`` = tokens with any flagged visit on the oracle
   path; ``n_path_divergent`` = tokens whose device path differs anywhere.
3. Values.  Per token, the raw normwise error
       err_b = ||y_dev - y_ref||_2 / ||y_ref||_2 <= tol,
   with y_ref evaluated in fp64 along the DEVICE path (tol = 1e-5 for fp32
   outputs, 2e-2 for bf16 outputs; for a bf16 output that adds to a base --
   residual or accumulate -- the error is taken on the stored total).
4. The one exception: ILL-CONDITIONED tokens, i.e. cancellation.  y_b is a
   sum over the visits v of act(l_v) W_out[n_v], and each logit l_v is itself
   a sum, of the H products x_i W_in[n_v, i].  Perturbing every input element
   and every product by a relative eps moves y_b by at most
   eps * kappa_b * ||y_b|| (to first order), with the componentwise condition
       kappa_b = sum_v (|act'(l_v)| S_v + |act(l_v)|) ||W_out[n_v]|| / ||y_b||,
       S_v = sum_i |x_i W_in[n_v, i]|.
   An fp32 evaluation that perturbs each input and product by no more than
   one unit roundoff u = 2^-24 (a backward-stable one) can therefore only
   promise u * kappa_b; when that exceeds the fp32 bar (kappa_b > KAPPA_MAX =
   1e-5 / u, about 168) the bar is not attainable in fp32 and the token is
   ill-conditioned.  kappa_b is large only under cancellation: a logit far
   smaller than the magnitudes it sums (|l_v| << S_v; at depth 0 the output
   is act(l) W_out[0], so a logit near 0 makes the whole output relatively
   inaccurate) or an output far below the sum of its terms (||y_b|| <<
   sum |act(l_v)| ||W_out[n_v]||).  Typical tokens of the depth-11, hidden-768
   layer have kappa_b around 50.  Only ill-conditioned tokens may exceed tol,
   and only by the first-order rounding bound of the fp32 arithmetic:
       allowance_b = sum_v [ |act'(l_v)| g_dot S_v
                             + (8 + l_v^2 + T(D+1) + 1) u |act(l_v)| ] ||W_out[n_v]||,
   g_dot = max(64, H/16 + 8) u bounding an fp32 dot product split over at
   least 16 lanes (a per-lane chain plus a reduction tree), 8 + l^2 the
   activation's own rounding (erfc's condition number near -l/sqrt 2), and
   T(D+1) + 1 the roundings of the output sum.  Tokens that used it are
   counted (``n_conditioned``) and a check fails when there are more than
   ``max_conditioned`` of them (0 unless the caller names a reason).
5. bf16 outputs, elementwise: every stored element lies within one bf16
   spacing of the fp64 value (base + y_ref) plus the fp32 bar 1e-5 ||y_ref||
   (plus the allowance for ill-conditioned tokens).  Rounding an fp32 result
   that meets the fp32 bar moves it by half a spacing at most (a whole one
   where it crosses into the next binade), so any error beyond fp32
   accumulation -- a dropped term, a coarser activation split -- shows.

Elementwise relative error is meaningless near zero, hence the normwise form;
the largest elementwise error scaled by ||y_ref||_inf is reported too.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erfc

from . import DEFAULT_TIE_REL, eval_path

U32 = 2.0 ** -24          # fp32 unit roundoff
FP32_BAR = 1e-5           # per-token normwise bar of an fp32 output
KAPPA_MAX = FP32_BAR / U32


def dot_gamma(hidden: int) -> float:
    """First-order bound, in units of ||x|| ||w||, on the rounding of an fp32 dot product of length
    hidden split over at least 16 lanes: a per-lane chain of hidden/16 terms plus a reduction tree."""
    return max(64.0, hidden / 16.0 + 8.0) * U32


def widen(a: np.ndarray) -> np.ndarray:
    """float32 or bf16-bit-pattern (uint16) array -> float64, exactly."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def _row_norm(w: np.ndarray, t: int, n: int) -> float:
    return float(np.linalg.norm(widen(w[t, n])))


def row_norms(w: np.ndarray, chunk: int = 4096) -> np.ndarray:
    """||row||_2 of every [T, N, H] weight row, as float64 [T, N] (chunked to bound memory)."""
    T, N, _ = w.shape
    out = np.empty((T, N))
    for t in range(T):
        for n0 in range(0, N, chunk):
            out[t, n0:n0 + chunk] = np.linalg.norm(widen(w[t, n0:n0 + chunk]), axis=1)
    return out


def _is_identity(act) -> bool:
    return act in ("identity", 2)


def _is_tanh(act) -> bool:
    return act in ("gelu_tanh", 1)


def act_values(z: np.ndarray, act) -> np.ndarray:
    """act(z) in float64: GELU z Phi(z) = z/2 erfc(-z/sqrt 2), its tanh form, or the identity."""
    z = np.asarray(z, dtype=np.float64)
    if _is_identity(act):
        return z.copy()
    if _is_tanh(act):
        u = math.sqrt(2.0 / math.pi) * (z + 0.044715 * z ** 3)
        return z / (1.0 + np.exp(-2.0 * u))
    return 0.5 * z * erfc(-z / math.sqrt(2.0))


def act_slope(logits: np.ndarray, act) -> np.ndarray:
    """|d act / d l| at the given logits (GELU: Phi(l) + l phi(l); identity: 1)."""
    z = np.asarray(logits, dtype=np.float64)
    if _is_identity(act):
        return np.ones_like(z)
    if _is_tanh(act):
        u = math.sqrt(2.0 / math.pi) * (z + 0.044715 * z ** 3)
        s = 1.0 / (1.0 + np.exp(-2.0 * u))
        sm = 1.0 / (1.0 + np.exp(2.0 * u))
        return np.abs(s + 2.0 * z * s * sm * math.sqrt(2.0 / math.pi) * (1.0 + 3 * 0.044715 * z * z))
    cdf = 0.5 * erfc(-z / math.sqrt(2.0))
    pdf = np.exp(-0.5 * z * z) / math.sqrt(2.0 * math.pi)
    return np.abs(cdf + z * pdf)


def dot_magnitudes(x_rows, w_in, nodes, chunk: int = 2048) -> np.ndarray:
    """S[b, t, l] = sum_i |x[b, i] W_in[t, nodes[b, t, l], i]|, float64 (chunked over tokens)."""
    x_rows = np.asarray(x_rows)
    B = x_rows.shape[0]
    T = w_in.shape[0]
    nodes = np.asarray(nodes).reshape(B, T, -1)
    out = np.empty(nodes.shape)
    for b0 in range(0, B, chunk):
        xa = np.abs(widen(x_rows[b0:b0 + chunk]))
        for t in range(T):
            rows = np.abs(widen(w_in[t][nodes[b0:b0 + chunk, t]]))  # [b, D+1, H]
            out[b0:b0 + chunk, t] = np.einsum("bh,blh->bl", xa, rows)
    return out


def conditioning(x_rows, w_in, w_out, depth: int, n_trees: int, nodes, logits, y_ref, act):
    """Per token: kappa_b (rule 4) and the allowance of rule 4, both float64 [B]."""
    B = y_ref.shape[0]
    H = np.asarray(x_rows).shape[1]
    nout = row_norms(w_out)
    tidx = np.arange(n_trees)[None, :, None]
    nodes = np.asarray(nodes).reshape(B, n_trees, depth + 1)
    l = np.asarray(logits, dtype=np.float64).reshape(B, n_trees, depth + 1)
    a = act_values(l, act)
    s = act_slope(l, act)
    S = dot_magnitudes(x_rows, w_in, nodes)
    wo = nout[tidx, nodes]
    ynorm = np.linalg.norm(y_ref, axis=1)
    terms = ((s * S + np.abs(a)) * wo).reshape(B, -1).sum(axis=1)
    with np.errstate(divide="ignore", invalid="ignore"):
        kappa = np.where(ynorm > 0, terms / np.maximum(ynorm, 1e-300), np.where(terms > 0, np.inf, 0.0))
    n_sum = n_trees * (depth + 1) + 1
    allow = (s * dot_gamma(H) * S + (8.0 + l * l + n_sum) * U32 * np.abs(a)) * wo
    return kappa, allow.reshape(B, -1).sum(axis=1)


def bf16_spacing(r: np.ndarray) -> np.ndarray:
    """Distance between consecutive bf16 values at |r|: 2^(e-8) for |r| in [2^(e-1), 2^e), floored at
    the subnormal step 2^-133."""
    _, e = np.frexp(np.asarray(r, dtype=np.float64))
    return np.ldexp(1.0, np.maximum(e - 8, -133))


def check(x, w_in, w_out, depth: int, n_trees: int, oracle_out: dict, y_dev, nodes_dev=None,
          tol: float = 1e-5, act="gelu", tie_rel: float = DEFAULT_TIE_REL, rows=None,
          base_dev=None, max_conditioned: int = 0) -> dict:
    """Compare device results with the oracle (rules in the module docstring).

    ``rows``: optional token indices the oracle output covers (sampled check);
    ``x`` and the device arrays are then indexed by it.  ``base_dev``: an
    optional [B,H] term the device added to FFF(x) (residual or accumulate),
    subtracted before comparing.
    """
    y_is_bf16 = np.asarray(y_dev).dtype == np.uint16
    y_dev = widen(y_dev)
    base = None
    if base_dev is not None:
        base = widen(base_dev)
        y_dev = y_dev - base
    if rows is not None:
        rows = np.asarray(rows)
        y_dev = y_dev[rows]
        if base is not None and base.shape[0] != y_dev.shape[0]:
            base = base[rows]
        x_rows = np.asarray(x)[rows]
        if nodes_dev is not None:
            nodes_dev = np.asarray(nodes_dev)[rows]
    else:
        x_rows = np.asarray(x)
    y_ref = oracle_out["y"].copy()
    nodes_ref = oracle_out["nodes"].copy()
    logits_ref = oracle_out["logits"].copy()
    nodes_or = oracle_out["nodes"]
    tie_or = oracle_out["near_tie"]
    B = y_ref.shape[0]
    report = {"tokens": int(B), "n_near_tie": int(tie_or.reshape(B, -1).any(axis=1).sum()),
              "n_path_divergent": 0, "path_failures": [], "value_failures": []}

    if nodes_dev is not None:
        nodes_dev = np.asarray(nodes_dev).reshape(nodes_or.shape)
        diverged = np.nonzero((nodes_dev != nodes_or).reshape(B, -1).any(axis=1))[0]
        report["n_path_divergent"] = int(diverged.size)
        for b in diverged:
            xb = x_rows[b]
            ok = True
            for t in range(n_trees):
                pd, po = nodes_dev[b, t], nodes_or[b, t]
                if np.array_equal(pd, po):
                    continue
                first = int(np.nonzero(pd != po)[0][0])
                if first == 0 or not tie_or[b, t, first - 1]:
                    ok = False
                    report["path_failures"].append((int(b), t, first, "diverged at a non-tie"))
                    break
            if not ok:
                continue
            try:
                y_path, logits_path = eval_path(xb, w_in, w_out, depth, n_trees, nodes_dev[b], act)
            except ValueError:
                report["path_failures"].append((int(b), -1, -1, "illegal device path"))
                continue
            xnorm = float(np.linalg.norm(widen(xb)))
            for t in range(n_trees):
                pd = nodes_dev[b, t]
                for level in range(depth):
                    logit = logits_path[t, level]
                    want = 2 * int(pd[level]) + 1 + (1 if logit > 0 else 0)
                    if int(pd[level + 1]) != want:
                        thresh = tie_rel * xnorm * _row_norm(w_in, t, int(pd[level]))
                        if not abs(logit) < thresh:
                            ok = False
                            report["path_failures"].append((int(b), t, level, "wrong sign off-tie"))
                            break
                if not ok:
                    break
            if ok:
                y_ref[b] = y_path
                nodes_ref[b] = nodes_dev[b]
                logits_ref[b] = logits_path

    kappa, allowance = conditioning(x_rows, w_in, w_out, depth, n_trees, nodes_ref, logits_ref, y_ref, act)
    ill = kappa > KAPPA_MAX
    allowance = np.where(ill, allowance, 0.0)
    # the compared quantity: the FFF output, or for a bf16 output on a base the stored total
    on_total = y_is_bf16 and base is not None
    cmp_dev = y_dev + base if on_total else y_dev
    cmp_ref = y_ref + base if on_total else y_ref
    diff = np.linalg.norm(cmp_dev - cmp_ref, axis=1)
    ref = np.linalg.norm(cmp_ref, axis=1)
    err = diff / np.maximum(ref, 1e-30)
    err[(ref == 0) & (diff == 0)] = 0.0
    conditioned = ill & (err > tol) & (diff <= tol * ref + allowance)
    report["n_ill_conditioned"] = int(ill.sum())
    report["max_kappa"] = float(kappa.max()) if B else 0.0
    report["n_conditioned"] = int(conditioned.sum())
    report["max_normwise_err_raw"] = float(err.max()) if B else 0.0
    skip = np.zeros(B, dtype=bool)
    if nodes_dev is None:
        # Without device paths a near-tie token may have branched the other way; skip those.
        skip = tie_or.reshape(B, -1).any(axis=1)
        report["n_skipped_near_tie"] = int(skip.sum())
    judged = np.where(conditioned | skip, 0.0, err)
    amax = np.max(np.abs(y_ref), axis=1)
    elem = np.max(np.abs(y_dev - y_ref), axis=1) / np.maximum(amax, 1e-30)
    report["max_normwise_err"] = float(np.where(skip, 0.0, err).max()) if B else 0.0
    report["max_elem_err_over_inf"] = float(np.where(skip, 0.0, elem).max()) if B else 0.0
    bad = np.nonzero(judged > tol)[0]
    report["value_failures"] = [(int(b), float(err[b])) for b in bad[:20]]
    report["n_value_failures"] = int(bad.size)
    elem_ok = True
    if y_is_bf16:
        total_ref = y_ref + (base if base is not None else 0.0)
        total_dev = y_dev + (base if base is not None else 0.0)
        bound = bf16_spacing(total_ref) + (FP32_BAR * np.linalg.norm(y_ref, axis=1) + allowance)[:, None]
        excess = np.max(np.abs(total_dev - total_ref) / bound, axis=1)
        excess = np.where(skip, 0.0, excess)
        report["bf16_elem_excess"] = float(excess.max()) if B else 0.0
        ebad = np.nonzero(excess > 1.0)[0]
        report["n_bf16_elem_failures"] = int(ebad.size)
        report["bf16_elem_failures"] = [(int(b), float(excess[b])) for b in ebad[:20]]
        elem_ok = ebad.size == 0
    report["ok"] = ((not report["path_failures"]) and bad.size == 0 and elem_ok
                    and report["n_conditioned"] <= max_conditioned)
    return report


def summary(rep: dict) -> str:
    """One line with the figures every parity check prints: raw error, conditioning counts, paths."""
    s = (f"max normwise err {rep['max_normwise_err_raw']:.2e} (raw), conditioned {rep['n_conditioned']} "
         f"of {rep['n_ill_conditioned']} ill-conditioned (max kappa {rep['max_kappa']:.1f}), "
         f"near-tie {rep['n_near_tie']}, divergent {rep['n_path_divergent']}")
    if "bf16_elem_excess" in rep:
        s += f", bf16 elementwise excess {rep['bf16_elem_excess']:.2f}"
    return s


def assert_parity(*args, **kwargs) -> dict:
    rep = check(*args, **kwargs)
    if not rep["ok"]:
        raise AssertionError(
            f"parity failed: {len(rep['path_failures'])} path failures "
            f"(first: {rep['path_failures'][:3]}), {rep['n_value_failures']} value failures "
            f"(first: {rep['value_failures'][:3]}), {rep.get('n_bf16_elem_failures', 0)} bf16 elementwise "
            f"failures (first: {rep.get('bf16_elem_failures', [])[:3]}); {summary(rep)}")
    return rep


def bf16_total_excess(y_dev_bits: np.ndarray, total_ref: np.ndarray, fff_ref: np.ndarray, tol: float) -> float:
    """Check of a bf16 output that stores a residual sum x + FFF(u), per element.

    The device stores the rounding of x + f_dev with f_dev within the FFF bar
    of the exact f (||f_dev - f|| <= tol ||f||, per token), so every element
    lies within one bf16 spacing of the fp64 total r = x + f plus tol ||f||:
    the rounding moves it by at most half a spacing at the fp32 sum, and the
    FFF error by at most its norm.  Spacing at r: 2^(e-8) for |r| in
    [2^(e-1), 2^e), floored at the subnormal step 2^-133.  Returns the worst
    ratio of the error to that bound (must be <= 1).
    """
    d = widen(y_dev_bits)
    r = np.asarray(total_ref, dtype=np.float64)
    if r.size == 0:
        return 0.0
    _, e = np.frexp(r)
    spacing = np.ldexp(1.0, np.maximum(e - 8, -133))
    bound = spacing + tol * np.linalg.norm(np.asarray(fff_ref, dtype=np.float64), axis=1, keepdims=True)
    return float(np.max(np.abs(d - r) / bound))



def _act_grad_np(z, act):
    from . import activation_grad
    return np.vectorize(lambda v: activation_grad(float(v), act), otypes=[float])(z)


def _act_np(z, act):
    from . import activation
    return np.vectorize(lambda v: activation(float(v), act), otypes=[float])(z)


def backward_check(x, w_in, w_out, depth: int, n_trees: int, dy, path, logits_given, dev: dict, ref: dict,
                   act="gelu", chunk: int = 2048) -> dict:
    """Compare a device backward with the oracle's (both along ``path`` [B,T,D+1]).

    Bounds are first order in the fp32 unit roundoff u and hold for ANY
    summation order (atomics included): a sum of n terms computed in fp32 is
    within (n-1) u sum|terms| of the exact one, and each term carries the error
    of its coefficient:
      a  = act(l):  |a_dev - a| <= |act'(l)| |l_given - l| + (8 + l^2) u |a|
      dl = da act'(l), da = <dy, W_out[n]> (an fp32 dot):
            |dl_dev - dl| <= |act'(l)| 64u ||dy|| ||W_out[n]|| + |da| e_g,
            e_g = 0.8 |l_given - l| + (16 + l^2) u (Phi(l) + |l| phi(l))
      The l^2 terms are erfc's condition number at -l/sqrt2 (about l^2 for
      large |l|) applied to the rounding of its argument; e_g is absolute
      because act' crosses zero; 0.8 bounds |act''| for GELU (the identity
      has act'' = 0 and exact coefficients).
    Per dW row: ||err|| <= sum_b [(n_row + 1) u |c_b| + e_b] ||v_b||  (v = dy or x);
    per dx row: ||err|| <= sum_visits [(T(D+1) + 1) u |dl| + e_dl] ||W_in[n]||.
    Also reports the largest error relative to sum_b |c_b| ||v_b|| (the scale
    of the terms) and to the bound.
    """
    B, H = np.asarray(dy).shape
    T, D = n_trees, depth
    N = (1 << (D + 1)) - 1
    xw = widen(x)
    gw = widen(dy)
    wi = w_in
    wo = w_out
    path = np.asarray(path).reshape(B, T, D + 1)
    lg = np.asarray(logits_given, dtype=np.float64).reshape(B, T, D + 1)
    s_out = np.zeros((T, N))
    s_in = np.zeros((T, N))
    b_out = np.zeros((T, N))
    b_in = np.zeros((T, N))
    cnt = np.zeros((T, N))
    b_dx = np.zeros(B)
    xn = np.linalg.norm(xw, axis=1)
    gn = np.linalg.norm(gw, axis=1)
    nwi, nwo = row_norms(wi), row_norms(wo)
    for t in range(T):
        np.add.at(cnt[t], path[:, t, :].reshape(-1), 1.0)
    for b0 in range(0, B, chunk):
        b1 = min(B, b0 + chunk)
        for t in range(T):
            nd = path[b0:b1, t, :]                            # [b, D+1]
            rows_i = widen(wi[t][nd])                         # [b, D+1, H]
            rows_o = widen(wo[t][nd])
            l64 = np.einsum("bh,blh->bl", xw[b0:b1], rows_i)
            da = np.einsum("bh,blh->bl", gw[b0:b1], rows_o)
            g = _act_grad_np(l64, act)
            a = _act_np(l64, act)
            dl = da * g
            dlg = np.abs(lg[b0:b1, t] - l64)
            if act in ("identity", 2):
                e_a = np.abs(g) * dlg
                e_g = np.zeros_like(l64)
            else:
                pdf = np.exp(-0.5 * l64 * l64) / math.sqrt(2.0 * math.pi)
                cdf = 0.5 * (1.0 + np.vectorize(math.erf, otypes=[float])(l64 / math.sqrt(2.0)))
                e_a = np.abs(g) * dlg + (8 + l64 * l64) * U32 * np.abs(a)
                e_g = 0.8 * dlg + (16 + l64 * l64) * U32 * (cdf + np.abs(l64) * pdf)
            e_dl = np.abs(g) * 64 * U32 * gn[b0:b1, None] * nwo[t][nd] + np.abs(da) * e_g
            n_row = cnt[t][nd]
            co = ((n_row + 1) * U32 * np.abs(a) + e_a) * gn[b0:b1, None]
            ci = ((n_row + 1) * U32 * np.abs(dl) + e_dl) * xn[b0:b1, None]
            np.add.at(b_out[t], nd.reshape(-1), co.reshape(-1))
            np.add.at(b_in[t], nd.reshape(-1), ci.reshape(-1))
            np.add.at(s_out[t], nd.reshape(-1), (np.abs(a) * gn[b0:b1, None]).reshape(-1))
            np.add.at(s_in[t], nd.reshape(-1), (np.abs(dl) * xn[b0:b1, None]).reshape(-1))
            b_dx[b0:b1] += (((T * (D + 1) + 1) * U32 * np.abs(dl) + e_dl) * nwi[t][nd]).sum(axis=1)
    rep = {"ok": True, "fail": []}
    for name, bound, scale in (("dw_out", b_out, s_out), ("dw_in", b_in, s_in)):
        if dev.get(name) is None:
            continue
        err = np.linalg.norm(widen(dev[name]) - ref[name], axis=2)
        visited = cnt > 0
        if np.any(widen(dev[name])[~visited] != 0):
            rep["ok"] = False
            rep["fail"].append(f"{name}: non-zero rows off every path")
        bad = visited & (err > bound * 1.0000001)
        if bad.any():
            rep["ok"] = False
            tt, nn = np.argwhere(bad)[0]
            rep["fail"].append(f"{name}: {int(bad.sum())} rows past the bound, e.g. ({tt},{nn}) "
                               f"err {err[tt, nn]:.3e} bound {bound[tt, nn]:.3e}")
        rel = err[visited] / np.maximum(scale[visited], 1e-300)
        rep[name + "_max_err_over_scale"] = float(rel.max()) if rel.size else 0.0
        frac = err[visited] / np.maximum(bound[visited], 1e-300)
        rep[name + "_max_err_over_bound"] = float(frac.max()) if frac.size else 0.0
    if dev.get("dx") is not None:
        err = np.linalg.norm(widen(dev["dx"]) - ref["dx"], axis=1)
        bound = b_dx.copy()
        if np.asarray(dev["dx"]).dtype == np.uint16:  # stored in bf16: half a spacing per element on top
            bound += 2.0 ** -9 * np.linalg.norm(ref["dx"], axis=1) * 1.01
        bad = err > bound * 1.0000001
        if bad.any():
            rep["ok"] = False
            b = int(np.nonzero(bad)[0][0])
            rep["fail"].append(f"dx: {int(bad.sum())} tokens past the bound, e.g. {b} err {err[b]:.3e} "
                               f"bound {bound[b]:.3e}")
        rep["dx_max_err_over_norm"] = float((err / np.maximum(np.linalg.norm(ref["dx"], axis=1), 1e-300)).max())
    return rep
