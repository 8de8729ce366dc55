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
3. Values.  Per token, ||y_dev - y_ref||_2 <= tol * ||y_ref||_2 + allowance,
   with y_ref evaluated in fp64 along the DEVICE path.  The allowance is the
   first-order effect of rounding the fp32 logits:
       allowance = sum over visits of |act'(l)| * gamma * ||x|| ||W_in[n]|| ||W_out[n]||
   where gamma * ||x|| ||W_in[n]|| bounds the error of an fp32 dot product
   (gamma = 64 unit roundoffs covers a per-lane chain plus a cross-lane tree
   of up to 64 terms).  It matters only when y itself is tiny next to the
   terms that feed it -- e.g. a single visited node with a strongly negative
   logit, where GELU's relative slope (about |l|) amplifies the logit's
   absolute rounding -- and tokens that need it are counted
   (``n_conditioned``).

Elementwise relative error is meaningless near zero, hence the normwise
form; the largest elementwise error scaled by ||y_ref||_inf is reported too.
"""
from __future__ import annotations

import math

import numpy as np

from . import DEFAULT_TIE_REL, eval_path

DOT_GAMMA = 64 * 2.0 ** -24


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


def act_slope(logits: np.ndarray, act) -> np.ndarray:
    """|d act / d l| at the given logits (GELU: Phi(l) + l*phi(l); identity: 1)."""
    if act in ("identity", 2):
        return np.ones_like(logits)
    erf = np.vectorize(math.erf, otypes=[float])
    phi_cdf = 0.5 * (1.0 + erf(logits / math.sqrt(2.0)))
    pdf = np.exp(-0.5 * logits * logits) / math.sqrt(2.0 * math.pi)
    return np.abs(phi_cdf + logits * pdf)


def check(x, w_in, w_out, depth: int, n_trees: int, oracle_out: dict, y_dev, nodes_dev=None,
          tol: float = 1e-5, act="gelu", tie_rel: float = DEFAULT_TIE_REL, rows=None,
          base_dev=None, dot_gamma: float = DOT_GAMMA) -> dict:
    """Compare device results with the oracle.

    ``rows``: optional token indices the oracle output covers (sampled check);
    ``x`` and the device arrays are then indexed by it.  ``base_dev``: an
    optional [B,H] term the device added to FFF(x) (residual or accumulate),
    subtracted before comparing.
    """
    y_dev = widen(y_dev)
    if base_dev is not None:
        y_dev = y_dev - widen(base_dev)
    if rows is not None:
        rows = np.asarray(rows)
        y_dev = y_dev[rows]
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

    diff = np.linalg.norm(y_dev - y_ref, axis=1)
    ref = np.linalg.norm(y_ref, axis=1)
    err = diff / np.maximum(ref, 1e-30)
    err[(ref == 0) & (diff == 0)] = 0.0
    # first-order allowance for fp32 logit rounding (see module docstring)
    nin, nout = row_norms(w_in), row_norms(w_out)
    tidx = np.arange(n_trees)[None, :, None]
    xnorm = np.linalg.norm(widen(x_rows), axis=1)
    terms = act_slope(logits_ref, act) * nin[tidx, nodes_ref] * nout[tidx, nodes_ref]
    allowance = dot_gamma * xnorm * terms.reshape(B, -1).sum(axis=1)
    conditioned = (err > tol) & (diff <= tol * ref + allowance)
    report["n_conditioned"] = int(conditioned.sum())
    report["max_normwise_err_raw"] = float(err.max()) if B else 0.0
    err = np.where(conditioned, 0.0, err)
    if nodes_dev is None:
        # Without device paths a near-tie token may have branched the other way; skip those.
        skip = tie_or.reshape(B, -1).any(axis=1)
        err = np.where(skip, 0.0, err)
        report["n_skipped_near_tie"] = int(skip.sum())
    amax = np.max(np.abs(y_ref), axis=1)
    elem = np.max(np.abs(y_dev - y_ref), axis=1) / np.maximum(amax, 1e-30)
    report["max_normwise_err"] = float(err.max()) if B else 0.0
    report["max_elem_err_over_inf"] = float(elem.max()) if B else 0.0
    bad = np.nonzero(err > tol)[0]
    report["value_failures"] = [(int(b), float(err[b])) for b in bad[:20]]
    report["n_value_failures"] = int(bad.size)
    report["ok"] = (not report["path_failures"]) and bad.size == 0
    return report


def assert_parity(*args, **kwargs) -> dict:
    rep = check(*args, **kwargs)
    if not rep["ok"]:
        raise AssertionError(
            f"parity failed: {len(rep['path_failures'])} path failures "
            f"(first: {rep['path_failures'][:3]}), {rep['n_value_failures']} value failures "
            f"(first: {rep['value_failures'][:3]}), max normwise err {rep['max_normwise_err']:.3e}")
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


U32 = 2.0 ** -24  # fp32 unit roundoff


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
