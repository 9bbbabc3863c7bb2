"""Pins for the oracle's DPB layer gradient (§2.2: normalized reconstruction
and the variance auxiliary loss around encode / decode).

The oracle composes the layer backward from its parts (normalize_bwd,
decode_bwd, variance-loss gradient, decode).  Here the same layer is written
as explicit matrices on the CPU — Phi_S stacked from single directions, coef
= Phi_S x with the indices held fixed, u = Phi_S^T coef, y = u ||x|| / ||u||,
and the loss <gy, y> + gloss * L_var(coef) with torch's population variance —
and differentiated by float64 autograd.  A dropped term (the norm path into
x, the auxiliary path into coef, the auxiliary term's decode into x) or a
wrong sign fails one of the comparisons.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_20652_amd import inputs


def _phi_stack(d, m, idx):
    T, k = idx.shape
    P = np.zeros((T, k, d))
    for t in range(T):
        for s in range(k):
            if idx[t, s] >= 0:
                P[t, s] = oracle.phi(d, m, int(idx[t, s]))
    return torch.tensor(P)


def _torch_var_loss(idx, c, n_min):
    flat_i, flat_c = idx.reshape(-1), c.reshape(-1)
    terms = []
    for f in np.unique(flat_i):
        if f < 0:
            continue
        sel = torch.tensor(flat_i == f)
        if int(sel.sum()) >= n_min:
            terms.append(flat_c[sel].var(unbiased=False))
    if not terms:
        return c.sum() * 0.0
    return -torch.stack(terms).mean()


@pytest.mark.parametrize("normalized,gloss,n_min", [(True, 0.7, 3), (False, 1.3, 2), (True, 0.0, 1)])
def test_layer_backward_equals_autograd_of_explicit_layer(normalized, gloss, n_min):
    w = inputs.workload("tiny")
    nb, dl, K = oracle.hierarchy(w.d, w.n, w.levels, w.branching, w.beam, w.k)
    m, gens = oracle.masks(w.d, w.n), oracle.generators(nb, dl, 0)
    T = 24
    x = inputs.activations("tiny", T).double().numpy()
    gy = inputs.upstream_grad("tiny", T).double().numpy()
    idx, coef, _, _ = oracle.encode(w.d, m, nb, K, dl, gens, x)

    Phi = _phi_stack(w.d, m, idx)                        # [T, k, d]
    xt = torch.tensor(x, requires_grad=True)
    c = torch.einsum("tkd,td->tk", Phi, xt)
    c.retain_grad()
    # the encoder's coefficients are exactly Phi_S x (indices fixed)
    assert np.allclose(c.detach().numpy(), coef, rtol=1e-12, atol=1e-12)
    u = torch.einsum("tkd,tk->td", Phi, c)
    y = u * (xt.norm(dim=1, keepdim=True) / u.norm(dim=1, keepdim=True)) if normalized else u
    L = (torch.tensor(gy) * y).sum() + gloss * _torch_var_loss(idx, c, n_min)
    L.backward()

    gc, gx = oracle.layer_backward(w.d, m, idx, coef, x, gy, gloss, n_min, normalized)
    assert np.allclose(gc, c.grad.numpy(), rtol=1e-10, atol=1e-11)
    assert np.allclose(gx, xt.grad.numpy(), rtol=1e-10, atol=1e-11)


def test_standardized_layer_backward_equals_autograd():
    """With standardized coefficients coef = (Phi_S x - mu) r the gradient to
    x carries r on every slot."""
    w = inputs.workload("tiny")
    nb, dl, K = oracle.hierarchy(w.d, w.n, w.levels, w.branching, w.beam, w.k)
    m, gens = oracle.masks(w.d, w.n), oracle.generators(nb, dl, 0)
    N = 1 << w.n
    rng = np.random.default_rng(4)
    mu = (0.3 * rng.standard_normal(N)).astype(np.float32)
    r = rng.uniform(0.5, 2.0, N).astype(np.float32)
    T = 20
    x = inputs.activations("tiny", T).double().numpy()
    gy = inputs.upstream_grad("tiny", T).double().numpy()
    idx, coef, _, _ = oracle.encode_std(w.d, m, nb, K, dl, gens, x, mu, r)
    Phi = _phi_stack(w.d, m, idx)
    live = torch.tensor(idx >= 0)
    mus = torch.tensor(np.where(idx >= 0, mu[np.maximum(idx, 0)], 0.0).astype(np.float64))
    rs = np.where(idx >= 0, r[np.maximum(idx, 0)], 0.0).astype(np.float64)
    xt = torch.tensor(x, requires_grad=True)
    c = torch.where(live, (torch.einsum("tkd,td->tk", Phi, xt) - mus) * torch.tensor(rs), torch.zeros(()))
    c.retain_grad()
    u = torch.einsum("tkd,tk->td", Phi, c)
    y = u * (xt.norm(dim=1, keepdim=True) / u.norm(dim=1, keepdim=True))
    L = (torch.tensor(gy) * y).sum() + 0.8 * _torch_var_loss(idx, c, 2)
    L.backward()
    # level-0 coefficients are fp32 on the encoder side; the layer's are fp64
    assert np.allclose(c.detach().numpy(), coef, rtol=1e-6, atol=1e-6)
    gc, gx = oracle.layer_backward(w.d, m, idx, c.detach().numpy(), x, gy, 0.8, 2, True, r_slot=rs)
    assert np.allclose(gc, c.grad.numpy(), rtol=1e-10, atol=1e-11)
    assert np.allclose(gx, xt.grad.numpy(), rtol=1e-10, atol=1e-11)


def test_layer_forward_pieces_agree_with_explicit_layer():
    """decode + normalize of the encoder's code equals the explicit layer."""
    w = inputs.workload("tiny")
    nb, dl, K = oracle.hierarchy(w.d, w.n, w.levels, w.branching, w.beam, w.k)
    m, gens = oracle.masks(w.d, w.n), oracle.generators(nb, dl, 0)
    x = inputs.activations("tiny", 16).double().numpy()
    idx, coef, _, _ = oracle.encode(w.d, m, nb, K, dl, gens, x)
    Phi = _phi_stack(w.d, m, idx).numpy()
    u = np.einsum("tkd,tk->td", Phi, np.einsum("tkd,td->tk", Phi, x))
    y, norms = oracle.normalize(oracle.decode(w.d, m, idx, coef), x)
    assert np.allclose(y, u * (np.linalg.norm(x, axis=1) / np.linalg.norm(u, axis=1))[:, None], rtol=1e-12)
    assert np.allclose(norms[:, 0], np.linalg.norm(x, axis=1))
