"""Comparison rules between the HIP path and the CPU oracle.

Encode (AbsTopK over fp32 scores vs the oracle's fp64 scores):
  * level 0 scores are the coordinates themselves on both sides, so level 0
    must match exactly -- indices, order and coefficients, ties included;
  * at a hashed level l >= 1 the oracle's boundary margin
        m = (|s|_(K) - |s|_(K+1)) / |s|_(K)
    decides: if m >= NEAR_TIE the index SETS must be equal, the ORDER must be
    equal where the smallest gap between consecutive selected scores is
    >= NEAR_TIE, and coefficients are compared on matched indices;
  * if m < NEAR_TIE, fp32 rounding may legitimately swap the boundary pair,
    so from that level on the token is checked against its own parents
    instead (check_selection): the GPU's candidates are the distinct children
    of the GPU's parents, each rescored by the oracle in fp64; the GPU's
    selection must be distinct candidates, as many as the level keeps, no
    selected score below an unselected one by more than NEAR_TIE of the K-th
    score, its order by the GPU's own coefficients, and every coefficient
    within tol of the oracle's score of that index;
  * a coefficient passes when |gpu - ref| <= tol * |ref|.
Decode / backward: |gpu - ref| <= tol * max(|ref|, rms(ref row)).
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


def coef_err(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """|got - ref| / max(|ref|, rms of ref along the last axis), element by
    element (0 where got equals ref): the relative bar taken against the
    row's scale, as for decoded rows, with one token's coefficients of one
    level as the row.  A level that keeps every child also keeps scores near
    zero, whose fp32 sums cannot meet 1e-5 of their own magnitude."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    diff = np.abs(got - ref)
    rms = np.sqrt(np.mean(ref * ref, axis=-1, keepdims=True)) if ref.size else ref
    den = np.maximum(np.abs(ref), rms)
    return np.where(diff == 0, 0.0, diff / np.where(den == 0, 1e-300, den))


class EncodeCheck:
    """What check_selection needs to rescore a token's candidates with the
    oracle: the dictionary (d, row masks, generators per level), the compared
    rows of x (fp64 [T, d], the same rows as the codes), and the
    standardization statistics (fp32 mu and r per feature) when the code was
    encoded on standardized scores."""

    def __init__(self, d, masks, gens, x, mu=None, r=None):
        self.d, self.masks, self.gens = d, masks, gens
        self.x = np.ascontiguousarray(np.asarray(x, dtype=np.float64))
        self.mu = None if mu is None else np.asarray(mu, dtype=np.float32)
        self.r = None if r is None else np.asarray(r, dtype=np.float32)

    def scores(self, t, ids):
        import oracle
        s = oracle.scores(self.d, self.masks, self.x[t], ids)
        if self.mu is not None:
            s = (s - self.mu[ids].astype(np.float64)) * self.r[ids].astype(np.float64)
        return s


def check_selection(ctx, t, l, K, parents, sel_idx, sel_coef, tol):
    """The GPU's level-l selection of token t from its own level-(l-1)
    parents is a valid AbsTopK of the exact scores (see the module notes)."""
    par = parents[parents >= 0].astype(np.int64)
    cands = np.unique((par[:, None] ^ ctx.gens[l].astype(np.int64)[None, :]).reshape(-1))
    s = ctx.scores(t, cands)
    n_keep = min(K, cands.size)
    live = sel_idx >= 0
    assert live.sum() == n_keep, f"token {t} level {l}: {live.sum()} selected, {n_keep} expected"
    assert (~live[n_keep:]).all() and (sel_coef[~live] == 0).all(), f"token {t} level {l}: padding misplaced"
    si = sel_idx[live].astype(np.int64)
    assert np.unique(si).size == si.size, f"token {t} level {l}: repeated index"
    pos = np.searchsorted(cands, si)
    assert (pos < cands.size).all() and (cands[np.minimum(pos, cands.size - 1)] == si).all(), \
        f"token {t} level {l}: an index is no child of the token's parents"
    mag = np.abs(s)
    chosen = np.zeros(cands.size, dtype=bool)
    chosen[pos] = True
    kth = np.sort(mag)[::-1][n_keep - 1] if n_keep else 0.0
    if (~chosen).any() and chosen.any():
        gap = mag[~chosen].max() - mag[chosen].min()
        assert gap <= NEAR_TIE * kth, f"token {t} level {l}: selection off by {gap} (K-th score {kth})"
    err = coef_err(sel_coef[live], s[pos])
    assert err.max(initial=0.0) <= tol, f"token {t} level {l}: coefficient error {err.max()}"
    c = np.abs(np.asarray(sel_coef[live], dtype=np.float64))
    ordered = (c[:-1] > c[1:]) | ((c[:-1] == c[1:]) & (si[:-1] < si[1:]))
    assert ordered.all(), f"token {t} level {l}: slots not in (|coef| desc, index asc) order"
    return float(err.max(initial=0.0))


def compare_encode(active, idx_g, coef_g, idx_o, coef_o, margin_o, order_o, tol=TOL_F32, ctx=None):
    """Returns statistics; raises AssertionError on a parity failure.  ctx (an
    EncodeCheck) is needed when some (token, level) is a near-tie."""
    idx_g, coef_g = np.asarray(idx_g), np.asarray(coef_g, dtype=np.float64)
    T = idx_o.shape[0]
    exempt = np.zeros(T, dtype=bool)
    stats = {"tokens": T, "exempt_tokens": 0, "rescored_levels": 0, "order_checked": 0, "max_coef_rel": 0.0}
    slot = 0
    bases = np.cumsum([0] + list(active))
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
        err = coef_err(np.take_along_axis(gc, og, 1), np.take_along_axis(oc, oo, 1))
        err = np.where(gs < 0, 0.0, err)
        stats["max_coef_rel"] = max(stats["max_coef_rel"], float(err.max(initial=0.0)))
        assert err.max(initial=0.0) <= tol, f"level {l}: coefficient error {err.max()}"
        # near-ties: the GPU's own choice, from the GPU's own parents, rescored exactly
        for t in np.nonzero(exempt)[0]:
            assert ctx is not None, "a near-tie needs an EncodeCheck context to be verified"
            e = check_selection(ctx, int(t), l, K, idx_g[t, bases[l - 1]:bases[l]], idx_g[t, sl], coef_g[t, sl], tol)
            stats["max_coef_rel"] = max(stats["max_coef_rel"], e)
            stats["rescored_levels"] += 1
    stats["exempt_tokens"] = int(exempt.sum())
    return stats


def compare_dense(got, ref, tol):
    err = rel_err(got, ref)
    assert err.max(initial=0.0) <= tol, f"max relative error {err.max()} > {tol}"
    return float(err.max(initial=0.0))


def random_std_state(N, seed, scale=1.0):
    """A standardization state (mu, m2, r) of N features, fp32, with variances
    m2 - mu^2 drawn in [0.3, 3] and r the inverse deviation they imply."""
    import oracle
    rng = np.random.default_rng(seed)
    mu = (0.3 * scale * rng.standard_normal(N)).astype(np.float32)
    var = rng.uniform(0.3, 3.0, N)
    m2 = (var + mu.astype(np.float64) ** 2).astype(np.float32)
    r = oracle.std_r(mu.astype(np.float64), m2.astype(np.float64), 1e-6).astype(np.float32)
    return mu, m2, r
