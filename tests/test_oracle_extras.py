"""Pins for the oracle's normalized reconstruction, code edits and variance
auxiliary loss (§2.2 "Normalized Reconstruction", "Auxillary losses"; the
greedy feature editing of App. C.3).

Normalization: output norm equals the reference norm, the direction is the
decoder's, positive rescaling of the decoder output changes nothing, and the
hand-derived backward equals float64 autograd of the forward definition.
Edits: each candidate changes the decode by exactly the removed / added
terms (decode is linear in the code), and replacing every position in turn
reaches the target code.  Variance loss: a hand-worked example
(tests/golden), finite differences of the loss for the gradient, invariance
to a per-feature shift, quadratic scaling, and the n_min cut.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "variance_loss_example.json")


def _rows(T, d, seed):
    return np.random.default_rng(seed).standard_normal((T, d))


def test_normalize_matches_reference_norm_and_direction():
    u, r = _rows(16, 64, 1), _rows(16, 64, 2)
    y, norms = oracle.normalize(u, r)
    assert np.allclose(np.linalg.norm(y, axis=1), np.linalg.norm(r, axis=1), rtol=1e-13)
    cos = np.sum(y * u, axis=1) / (np.linalg.norm(y, axis=1) * np.linalg.norm(u, axis=1))
    assert np.allclose(cos, 1.0, atol=1e-13)
    assert np.allclose(norms[:, 0], np.linalg.norm(r, axis=1)) and np.allclose(norms[:, 1], np.linalg.norm(u, axis=1))
    y2, _ = oracle.normalize(3.5 * u, r)
    assert np.allclose(y2, y, rtol=1e-13, atol=1e-14)


def test_normalize_zero_output_row():
    u, r = _rows(4, 32, 3), _rows(4, 32, 4)
    u[1] = 0.0
    y, _ = oracle.normalize(u, r)
    assert np.all(y[1] == 0.0) and np.all(np.isfinite(y))
    g = _rows(4, 32, 5)
    gu, gr = oracle.normalize_bwd(g, u, r)
    assert np.all(gu[1] == 0.0) and np.all(gr[1] == 0.0)


def test_normalize_backward_equals_autograd():
    T, d = 8, 48
    u, r, g = _rows(T, d, 6), _rows(T, d, 7), _rows(T, d, 8)
    ut = torch.tensor(u, requires_grad=True)
    rt = torch.tensor(r, requires_grad=True)
    y = ut * (rt.norm(dim=1, keepdim=True) / ut.norm(dim=1, keepdim=True))
    (y * torch.tensor(g)).sum().backward()
    gu, gr = oracle.normalize_bwd(g, u, r)
    assert np.allclose(gu, ut.grad.numpy(), rtol=1e-12, atol=1e-13)
    assert np.allclose(gr, rt.grad.numpy(), rtol=1e-12, atol=1e-13)


@pytest.fixture(scope="module")
def tiny_code():
    d, n = 64, 12
    m = oracle.masks(d, n)
    rng = np.random.default_rng(9)
    T, k = 6, 10
    idx = rng.integers(0, 1 << n, size=(T, k)).astype(np.int32)
    idx[:, 0] = 7           # a basis feature everywhere
    idx[1, 5] = -1          # padding
    coef = rng.standard_normal((T, k))
    tidx = rng.integers(0, 1 << n, size=(T, k)).astype(np.int32)
    tcoef = rng.standard_normal((T, k))
    return d, m, idx, coef, tidx, tcoef


def test_edit_candidates_change_decode_by_exact_terms(tiny_code):
    """Decode is linear in the code, so each candidate's decode differs from
    its source row's by exactly the terms the edit removes and adds."""
    d, m, idx, coef, tidx, tcoef = tiny_code
    T, k = idx.shape
    base = oracle.decode(d, m, idx, coef)
    edits = [(r, p, op) for r in range(T) for p in (0, 3, 9) for op in range(4)]
    oi, oc = oracle.edit_codes(idx, coef, tidx, tcoef, edits)
    dec = oracle.decode(d, m, oi, oc)
    phi = lambda i: oracle.phi(d, m, int(i)) if i >= 0 else np.zeros(d)
    for e, (r, p, op) in enumerate(edits):
        old = coef[r, p] * phi(idx[r, p])
        if op == 0:
            expect = base[r] - old
        elif op == 1:
            expect = base[r] - old + tcoef[r, p] * phi(tidx[r, p])
        elif op == 2:
            expect = base[r] - old + tcoef[r, p] * phi(idx[r, p])
        else:
            expect = base[r]
        assert np.allclose(dec[e], expect, atol=1e-12), (r, p, op)
        other = np.arange(k) != p
        assert np.array_equal(oi[e, other], idx[r, other]) and np.array_equal(oc[e, other], coef[r, other])


def test_edit_out_of_range_gives_padding(tiny_code):
    _, _, idx, coef, tidx, tcoef = tiny_code
    T, k = idx.shape
    oi, oc = oracle.edit_codes(idx, coef, tidx, tcoef, [(T, 0, 0), (-1, 0, 0), (0, k, 0), (0, 0, 4), (0, 0, -1)])
    assert np.all(oi == -1) and np.all(oc == 0.0)


def test_edit_chain_reaches_target(tiny_code):
    """Replacing every position in turn turns the source code into the target."""
    _, _, idx, coef, tidx, tcoef = tiny_code
    ci, cc = idx[2:3].copy(), coef[2:3].copy()
    for p in range(idx.shape[1]):
        ci, cc = oracle.edit_codes(ci, cc, tidx[2:3], tcoef[2:3], [(0, p, 1)])
    assert np.array_equal(ci[0], tidx[2]) and np.array_equal(cc[0], tcoef[2])


def test_variance_loss_hand_example():
    ex = json.load(open(GOLDEN))
    loss, grad = oracle.variance_loss(np.array(ex["idx"]), np.array(ex["coef"]), ex["n_min"])
    assert loss == pytest.approx(ex["loss"], rel=1e-14)
    assert np.allclose(grad, np.array(ex["grad"]), rtol=1e-14, atol=1e-15)


def _random_code(seed, T=40, k=6, nfeat=12):
    rng = np.random.default_rng(seed)
    idx = rng.integers(0, nfeat, size=(T, k)).astype(np.int32)
    idx[rng.random((T, k)) < 0.1] = -1
    return idx, rng.standard_normal((T, k))


def test_variance_loss_gradient_finite_differences():
    idx, coef = _random_code(11)
    loss, grad = oracle.variance_loss(idx, coef, 5)
    h = 1e-6
    for t, s in [(0, 0), (3, 2), (17, 5), (39, 1)]:
        cp, cm = coef.copy(), coef.copy()
        cp[t, s] += h
        cm[t, s] -= h
        fd = (oracle.variance_loss(idx, cp, 5)[0] - oracle.variance_loss(idx, cm, 5)[0]) / (2 * h)
        assert fd == pytest.approx(grad[t, s], rel=1e-6, abs=1e-9)


def test_variance_loss_invariances():
    idx, coef = _random_code(12)
    loss, _ = oracle.variance_loss(idx, coef, 4)
    shifted = coef + np.where(idx == 3, 10.0, 0.0) - np.where(idx == 5, 4.0, 0.0)
    assert oracle.variance_loss(idx, shifted, 4)[0] == pytest.approx(loss, rel=1e-11)
    assert oracle.variance_loss(idx, 3.0 * coef, 4)[0] == pytest.approx(9.0 * loss, rel=1e-12)
    # n_min above every count: no feature qualifies
    assert oracle.variance_loss(idx, coef, 10 ** 6)[0] == 0.0
