"""Comparison rules between the HIP path and the CPU oracle.

Encode (AbsTopK over fp32 scores vs the oracle's fp64 scores):
  * level 0 scores are the coordinates themselves on both sides, so level 0
    must match exactly -- indices, order and coefficients, ties included;
  * at a hashed level l >= 1 the oracle's boundary margin
        m = (|s|_(K) - |s|_(K+1)) / |s|_(K)
    decides: if m < NEAR_TIE that (token, level) and every later level of the
    token are exempt (fp32 rounding may legitimately swap the boundary pair);
    otherwise the index SETS must be equal, the ORDER must be equal where the
    smallest gap between consecutive selected scores is >= NEAR_TIE, and
    coefficients are compared on matched indices;
  * a coefficient passes when |gpu - ref| <= tol * max(|ref|, rms(ref level row)).
Decode / backward: the same elementwise rule on every output, rms over the row.
"""
from __future__ import annotations

import numpy as np

NEAR_TIE = 1e-5
TOL_F32 = 1e-5
TOL_BF16 = 2e-2


def rel_err(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    rms = np.sqrt(np.mean(ref * ref, axis=-1, keepdims=True))
    den = np.maximum(np.abs(ref), rms)
    den = np.where(den == 0, 1.0, den)
    return np.abs(got - ref) / den


def compare_encode(active, idx_g, coef_g, idx_o, coef_o, margin_o, order_o, tol=TOL_F32):
    """Returns statistics; raises AssertionError on a parity failure."""
    idx_g, coef_g = np.asarray(idx_g), np.asarray(coef_g, dtype=np.float64)
    T = idx_o.shape[0]
    exempt = np.zeros(T, dtype=bool)
    stats = {"tokens": T, "exempt_tokens": 0, "order_checked": 0, "max_coef_rel": 0.0}
    slot = 0
    for l, K in enumerate(active):
        sl = slice(slot, slot + K)
        slot += K
        if l == 0:
            assert np.array_equal(idx_g[:, sl], idx_o[:, sl]), "level 0 indices differ"
            assert np.array_equal(coef_g[:, sl], coef_o[:, sl]), "level 0 coefficients differ"
            continue
        exempt |= margin_o[:, l] < NEAR_TIE
        live = ~exempt
        gi, oi = idx_g[live, sl], idx_o[live, sl]
        gc, oc = coef_g[live, sl], coef_o[live, sl]
        og = np.argsort(gi, axis=1, kind="stable")
        oo = np.argsort(oi, axis=1, kind="stable")
        gs = np.take_along_axis(gi, og, 1)
        os_ = np.take_along_axis(oi, oo, 1)
        bad = np.nonzero(np.any(gs != os_, axis=1))[0]
        assert bad.size == 0, f"level {l}: index sets differ on {bad.size} tokens, first {np.nonzero(live)[0][bad[0]]}"
        ordered = order_o[live, l] >= NEAR_TIE
        stats["order_checked"] += int(ordered.sum())
        assert np.array_equal(gi[ordered], oi[ordered]), f"level {l}: order differs"
        err = rel_err(np.take_along_axis(gc, og, 1), np.take_along_axis(oc, oo, 1))
        err = np.where(gs < 0, 0.0, err)
        stats["max_coef_rel"] = max(stats["max_coef_rel"], float(err.max(initial=0.0)))
        assert err.max(initial=0.0) <= tol, f"level {l}: coefficient error {err.max()}"
    stats["exempt_tokens"] = int(exempt.sum())
    return stats


def compare_dense(got, ref, tol):
    err = rel_err(got, ref)
    assert err.max(initial=0.0) <= tol, f"max relative error {err.max()} > {tol}"
    return float(err.max(initial=0.0))
