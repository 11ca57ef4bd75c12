"""Plant plausible mistakes in the oracle (on the CPU) and check that the pins
catch every one of them: a dropped term, a wrong sign, a transposed operand,
the wrong end of the spectrum, a missing normalisation."""
import types

import numpy as np
import pytest

import oracle
from oracle import espace_ref as R
from tests import oracle_pins


def _base():
    return {k: getattr(oracle, k) for k in dir(oracle) if not k.startswith("_")}


def _fold_transposed_p(W, Pt):
    # uses Pt as if it were P (K×L); only shape-valid when L == K
    return np.asarray(W, float) @ np.asarray(Pt, float)


def _project_drops_last(Pt, X):
    Z = R.project(Pt, X)
    Z[:, -1] = 0.0
    return Z


def _expand_sign(Z, Wf):
    return -R.expand(Z, Wf)


def _expand_transposed(Z, Wf):
    Z = np.asarray(Z, float)
    Wf = np.asarray(Wf, float)
    return (Z @ Wf.T)[:, ::-1].copy()


def _dense_transposed(X, W):
    return np.asarray(X, float) @ np.asarray(W, float)[::-1].T


def _pc_ascending(C, L):
    d, V = np.linalg.eigh(np.asarray(C, float))
    return np.ascontiguousarray(V[:, :L].T), d


def _autocorr_unscaled(batches):
    C = None
    for Xi in batches:
        Xi = np.asarray(Xi, float)
        Ci = Xi.T @ Xi
        C = Ci if C is None else C + Ci
    return C / len(batches)


def _autocorr_pooled(batches):
    X = np.concatenate([np.asarray(b, float) for b in batches])
    return X.T @ X / X.shape[0]


def _reconstruct_drops_term(Pt, X):
    return R.reconstruct(np.asarray(Pt)[:-1], X) if len(Pt) > 1 else 0 * np.asarray(X, float)


def _normalized_plain(batches):
    return R.autocorrelation(batches)


def _fold_skips_projection(W, Pt):
    W = np.asarray(W, float)
    L = len(Pt)
    return W[:, :L].copy()


def _gomse_one_sided(CX, CW):
    return np.asarray(CX, float) @ np.asarray(CW, float) * 2


def _by_value(C, L):
    return R.principal_components(C, L)


def _by_magnitude_ascending(C, L):
    d, V = np.linalg.eigh(np.asarray(C, float))
    order = np.argsort(np.abs(d), kind="stable")
    return np.ascontiguousarray(V[:, order[:L]].T), d[order]


def _train_bwd_no_projection(dY, X, Pt, W):
    dY = np.asarray(dY, float)
    W = np.asarray(W, float)
    Xt = R.reconstruct(Pt, X)
    return dY @ W, dY.T @ Xt


def _train_bwd_dw_raw_x(dY, X, Pt, W):
    dX, _ = R.train_backward(dY, X, Pt, W)
    return dX, np.asarray(dY, float).T @ np.asarray(X, float)


def _dense_bwd_transposed(dY, X, W):
    dX, dW = R.dense_backward(dY, X, W)
    return dX, dW[::-1].copy()


def _nlmse_pooled(pairs, normalized=False):
    X = np.concatenate([np.asarray(a, float) for a, _ in pairs])
    G = np.concatenate([np.asarray(b, float) for _, b in pairs])
    return R.nlmse_matrix([(X, G)], normalized)


def _nlmse_unnormalised(pairs, normalized=False):
    return R.nlmse_matrix(pairs, False)


MUTANTS = {
    "fold uses Pt for P": {"fold": _fold_transposed_p},
    "fold ignores P": {"fold": _fold_skips_projection},
    "project drops a component": {"project": _project_drops_last},
    "expand flips sign": {"expand": _expand_sign},
    "expand permutes outputs": {"expand": _expand_transposed},
    "dense permutes weights": {"dense": _dense_transposed},
    "smallest eigenvectors": {"principal_components": _pc_ascending},
    "autocorrelation without 1/M": {"autocorrelation": _autocorr_unscaled},
    "autocorrelation pooled, not batch-averaged": {"autocorrelation": _autocorr_pooled},
    "reconstruct drops a term": {"reconstruct": _reconstruct_drops_term},
    "normalised autocorrelation not normalised": {"normalized_autocorrelation": _normalized_plain},
    "GO-MSE matrix one-sided": {"gomse_matrix": _gomse_one_sided},
    "selection by value, not magnitude": {"principal_components_by_magnitude": _by_value},
    "selection by smallest magnitude": {"principal_components_by_magnitude": _by_magnitude_ascending},
    "training dX skips the projection": {"train_backward": _train_bwd_no_projection},
    "training dW from unprojected X": {"train_backward": _train_bwd_dw_raw_x},
    "dense dW rows permuted": {"dense_backward": _dense_bwd_transposed},
    "NL-MSE pooled across sequences": {"nlmse_matrix": _nlmse_pooled},
    "NL-MSE normalised variant not normalised": {"nlmse_matrix": _nlmse_unnormalised},
}


from oracle import mxfp8_ref as MX


def _e4m3_ties_away(v):
    v = np.asarray(v, dtype=np.float64)
    a = np.minimum(np.abs(v), 448.0)
    _, e = np.frexp(a)
    e = np.maximum(e - 1, -6)
    step = np.ldexp(1.0, e - 3)
    return np.copysign(np.minimum(np.floor(a / step + 0.5) * step, 448.0), v)


def _e4m3_no_clamp(v):
    v = np.asarray(v, dtype=np.float64)
    a = np.abs(v)
    _, e = np.frexp(a)
    e = np.maximum(e - 1, -6)
    step = np.ldexp(1.0, e - 3)
    return np.copysign(np.rint(a / step) * step, v)


def _mx_quantize_emax7(A):
    # S = floor(log2 amax) - 7: elements land in [128, 256), one bit lost
    q, sb = MX.mx_quantize(np.asarray(A, dtype=np.float64) / 2.0)
    sb = np.where(sb > 0, sb.astype(np.int64) + 1, 0).clip(0, 254).astype(np.uint8)
    return MX.e4m3_round(q / 2.0), sb


def _mx_quantize_block16(A):
    A = np.asarray(A, dtype=np.float64)
    rows, cols = A.shape
    q = np.zeros_like(A)
    sb = np.zeros((rows, -(-cols // 32)), np.uint8)
    for c0 in range(0, cols, 16):
        qq, ss = MX.mx_quantize(A[:, c0:c0 + 16])
        q[:, c0:c0 + 16] = qq
        if c0 % 32 == 0:
            sb[:, c0 // 32] = ss[:, 0]
    return q, sb


def _mx_layer_no_requant(Xq, Xs, Ptq, Pts, Wfq, Wfs):
    Z = MX.mx_project(Xq, Xs, Ptq, Pts)
    Zq, Zs = MX.mx_quantize(Z)
    return Z @ MX.mx_dequantize(Wfq, Wfs).T, Zq, Zs


def _mx_dequantize_no_scale(values, scale_bytes):
    return np.asarray(values, dtype=np.float64)


def _mx_expand_transposed_scales(Zq, Zs, Wfq, Wfs):
    return MX.mx_dequantize(Zq, Zs) @ (np.asarray(Wfq, float) * MX.mx_scale(Wfs[::-1], Wfq.shape[1])).T


MUTANTS.update({
    "e4m3 ties away from zero": {"e4m3_round": _e4m3_ties_away},
    "e4m3 without saturation": {"e4m3_round": _e4m3_no_clamp},
    "MX scale exponent off by one": {"mx_quantize": _mx_quantize_emax7},
    "MX blocks of 16": {"mx_quantize": _mx_quantize_block16},
    "MX layer skips re-quantising Z": {"mx_projected_linear": _mx_layer_no_requant},
    "MX dequantisation ignores scales": {"mx_dequantize": _mx_dequantize_no_scale},
    "MX expand uses another row's scales": {"mx_expand": _mx_expand_transposed_scales},
})


def _caught(ns):
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(ns)
        except Exception:
            return pin.__name__
    return None


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    fns = _base()
    fns.update(MUTANTS[name])
    if "fold" in MUTANTS[name] or "project" in MUTANTS[name] or "expand" in MUTANTS[name]:
        # keep the composed helpers consistent with the mutated step
        f, p, e = fns["fold"], fns["project"], fns["expand"]
        fns["projected_linear_from_weights"] = lambda X, Pt, W: e(p(Pt, X), f(W, Pt))
        fns["projected_linear"] = lambda X, Pt, Wf: e(p(Pt, X), Wf)
        fns["sampled_projected_linear"] = (
            lambda X, Pt, W, rows, cols: e(p(Pt, np.asarray(X)[rows]), f(np.asarray(W)[cols], Pt)))
    if "dense" in MUTANTS[name]:
        d = fns["dense"]
        fns["sampled_dense"] = lambda X, W, rows, cols: d(np.asarray(X)[rows], np.asarray(W)[cols])
    ns = types.SimpleNamespace(**fns)
    assert _caught(ns) is not None, f"mutant '{name}' passes every pin"
