"""Pins for the oracle's normalized reconstruction, code edits and variance
auxiliary loss (§2.2 "Normalized Reconstruction", "Auxillary losses"; the
feature-edit experiments of the appendix).

Normalization: output norm equals the reference norm, the direction is the
decoder's, positive rescaling of the decoder output changes nothing, and the
hand-derived backward equals float64 autograd of the forward definition.
Edits: each edit changes the decode by exactly the removed / added terms
(decode is linear in the code).  Variance loss: a hand-worked example
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
    idx[::2, 3] = 1234      # a hashed feature on even tokens
    idx[1, 5] = -1          # padding
    coef = rng.standard_normal((T, k))
    return d, m, idx, coef


def test_edit_zero_rescale_set_remove_exact_terms(tiny_code):
    d, m, idx, coef = tiny_code
    base = oracle.decode(d, m, idx, coef)
    contrib = lambda f, c: np.stack([sum(c[t, s] * oracle.phi(d, m, f) for s in range(idx.shape[1]) if idx[t, s] == f)
                                     if np.any(idx[t] == f) else np.zeros(d) for t in range(idx.shape[0])])
    for f in (7, 1234):
        i2, c2 = oracle.edit_codes(idx, coef, [(f, 0, 0.0, 0)])
        assert np.array_equal(i2, idx)
        assert np.allclose(oracle.decode(d, m, i2, c2), base - contrib(f, coef), atol=1e-12)
        i3, c3 = oracle.edit_codes(idx, coef, [(f, 1, 2.5, 0)])
        assert np.allclose(oracle.decode(d, m, i3, c3), base + 1.5 * contrib(f, coef), atol=1e-12)
        i4, c4 = oracle.edit_codes(idx, coef, [(f, 2, 0.75, 0)])
        ones = np.where(idx == f, 0.75, 0.0)
        assert np.allclose(oracle.decode(d, m, i4, c4), base - contrib(f, coef) + contrib(f, ones), atol=1e-12)


def test_edit_replace_moves_the_terms(tiny_code):
    d, m, idx, coef = tiny_code
    base = oracle.decode(d, m, idx, coef)
    i2, c2 = oracle.edit_codes(idx, coef, [(1234, 3, 0.0, 2048)])
    assert np.array_equal(c2, coef) and not np.any(i2 == 1234)
    w = np.where(idx == 1234, coef, 0.0).sum(axis=1, keepdims=True)
    expect = base + w * (oracle.phi(d, m, 2048) - oracle.phi(d, m, 1234))[None, :]
    assert np.allclose(oracle.decode(d, m, i2, c2), expect, atol=1e-12)


def test_edits_apply_in_order(tiny_code):
    _, _, idx, coef = tiny_code
    i2, c2 = oracle.edit_codes(idx, coef, [(1234, 3, 0.0, 99), (99, 1, -2.0, 0)])
    assert np.allclose(c2[idx == 1234], -2.0 * coef[idx == 1234])


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
