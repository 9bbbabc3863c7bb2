"""Pins for the oracle's encoder, decoder and decoder backward.

Encode: with full generator sets every parent reaches the whole next level, so
the beam search must equal brute-force per-level AbsTopK over a materialised
dense dictionary (the hierarchy of §2.2 then prunes nothing).  Inputs with
many exact ties exercise the (|s| desc, index asc) rule and DAG dedup.
Decode / backward: dense matrix products, exact dyadic linearity, float64
autograd through a dense Phi_S, and the adjoint identity.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2607_20652_amd import inputs


def dense_dictionary(d, m, N):
    """Phi [N, d] from §2.1 Eqs. 1-2: e_i below d, (-1)^{popcount(M_iota & i)}/sqrt d above."""
    i = np.arange(N, dtype=np.uint32)[:, None]
    par = np.bitwise_count(m[None, :] & i) & 1
    Phi = np.where(par == 1, -1.0, 1.0) / math.sqrt(d)
    Phi[:d] = np.eye(d)
    return Phi


def abstopk(scores, ids, K):
    order = np.lexsort((ids, -np.abs(scores)))  # |s| desc, then index asc
    return ids[order[:K]], scores[order[:K]]


def brute_force_levels(x, Phi, ranges, K):
    out_i, out_c = [], []
    for (lo, hi), k in zip(ranges, K):
        ids = np.arange(lo, hi)
        s = Phi[lo:hi] @ x
        i, c = abstopk(s, ids, k)
        out_i.append(i)
        out_c.append(c)
    return np.concatenate(out_i), np.concatenate(out_c)


TINY_FULL = dict(d=64, nbits=[6, 9, 12], K=[4, 4, 8])


def _full_gens(nbits):
    return [np.zeros(0, np.uint32)] + [np.arange(1 << nbits[l - 1], 1 << nbits[l], dtype=np.uint32)
                                       for l in range(1, len(nbits))]


@pytest.mark.parametrize("kind", ["normal", "dyadic"])
def test_beam_equals_brute_force_with_full_generators(kind):
    d, nbits, K = TINY_FULL["d"], TINY_FULL["nbits"], TINY_FULL["K"]
    m = oracle.masks(d, nbits[-1])
    gens = _full_gens(nbits)
    delta = [0] + [len(g) for g in gens[1:]]
    T = 64
    x = (inputs.activations("tiny", T) if kind == "normal" else inputs.dyadic(d, T)).double().numpy()
    idx, coef, _, _ = oracle.encode(d, m, nbits, K, delta, gens, x)
    Phi = dense_dictionary(d, m, 1 << nbits[-1])
    ranges = [(0, d)] + [(1 << nbits[l - 1], 1 << nbits[l]) for l in range(1, len(nbits))]
    for t in range(T):
        bi, bc = brute_force_levels(x[t], Phi, ranges, K)
        assert np.array_equal(idx[t], bi.astype(np.int32)), t
        assert np.allclose(coef[t], bc, rtol=0, atol=1e-12)


def test_dyadic_inputs_produce_exact_ties():
    """Control for the test above: the dyadic draw really has tied scores at the
    selection boundary, so the index tie-break is exercised."""
    d, nbits = 64, [6, 9, 12]
    m = oracle.masks(d, 12)
    x = inputs.dyadic(d, 64).double().numpy()
    Phi = dense_dictionary(d, m, 1 << 12)
    s = np.abs(Phi[512:4096] @ x.T)
    srt = -np.sort(-s, axis=0)
    assert (srt[7] == srt[8]).sum() > 10


def _beam_reference(x, Phi, d, nbits, K, gens):
    """Level-by-level candidate enumeration with numpy (independent of the C code)."""
    i0, c0 = abstopk(x[:d], np.arange(d), K[0])
    out_i, out_c, parents = [i0], [c0], i0
    for l in range(1, len(nbits)):
        cand = np.unique((parents[:, None] ^ gens[l][None, :].astype(np.int64)).ravel())
        s = Phi[cand] @ x
        il, cl = abstopk(s, cand, K[l])
        out_i.append(il)
        out_c.append(cl)
        parents = il
    return np.concatenate(out_i), np.concatenate(out_c)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_beam_with_sampled_generators_matches_numpy_enumeration(seed):
    d, n, L, b, B, k = 64, 12, 3, 16, 4, 8
    nbits, delta, K = oracle.hierarchy(d, n, L, b, B, k)
    assert (nbits, delta, K) == ([6, 9, 12], [0, 16, 16], [4, 4, 8])
    gens = oracle.generators(nbits, delta, seed)
    m = oracle.masks(d, n)
    Phi = dense_dictionary(d, m, 1 << n)
    x = inputs.activations("tiny", 48).double().numpy()
    idx, coef, margin, order = oracle.encode(d, m, nbits, K, delta, gens, x)
    for t in range(48):
        ri, rc = _beam_reference(x[t], Phi, d, nbits, K, gens)
        assert np.array_equal(idx[t], ri.astype(np.int32))
        assert np.allclose(coef[t], rc, atol=1e-12, rtol=0)
    assert (margin >= 0).all() and (order >= 0).all()


def test_dedup_is_needed():
    """Control: with these generators DAG duplicates do occur among candidates,
    and the oracle never emits an index twice."""
    d, nbits, delta, K = 64, [6, 9, 12], [0, 16, 16], [4, 4, 8]
    gens = oracle.generators(nbits, delta, 0)
    m = oracle.masks(d, 12)
    x = inputs.activations("tiny", 256).double().numpy()
    idx, _, _, _ = oracle.encode(d, m, nbits, K, delta, gens, x)
    for t in range(256):
        assert len(set(idx[t].tolist())) == idx.shape[1]
    dup = 0
    for t in range(256):
        par = idx[t, :4].astype(np.int64)
        c = (par[:, None] ^ gens[1][None, :].astype(np.int64)).ravel()
        dup += len(c) - len(np.unique(c))
    assert dup > 0


def test_padding_when_too_few_candidates():
    """Reading R7: fewer distinct candidates than K_l pads with (-1, 0)."""
    d, nbits, delta, K = 64, [6, 7], [0, 2], [1, 4]
    gens = [np.zeros(0, np.uint32), np.array([64, 65], np.uint32)]
    m = oracle.masks(d, 7)
    x = inputs.activations("tiny", 4).double().numpy()
    idx, coef, _, _ = oracle.encode(d, m, nbits, K, delta, gens, x)
    assert idx.shape[1] == 5                       # K_0 + K_1 slots
    assert (idx[:, 3:] == -1).all() and (coef[:, 3:] == 0).all()
    assert (idx[:, 1:3] >= 64).all()                # the two real candidates


def test_level0_matches_torch_topk_with_stable_ties():
    """Level 0 is AbsTopK of the coordinates themselves (§2.1 Eq. 2; the library
    routine torch.sort(stable=True) gives the index tie-break)."""
    d, nbits, delta, K = 768, [10, 12], [0, 16], [8, 8]
    m = oracle.masks(d, 12)
    gens = oracle.generators(nbits, delta, 0)
    x = inputs.activations("gpt2", 64)  # bf16: many exact ties
    idx, coef, _, _ = oracle.encode(d, m, nbits, K, delta, gens, x.double().numpy())
    xa = x.float().abs()
    order = torch.sort(-xa, dim=1, stable=True).indices[:, :8]
    assert np.array_equal(idx[:, :8], order.numpy().astype(np.int32))
    assert np.array_equal(coef[:, :8], torch.gather(x.double(), 1, order).numpy())


# ---------------------------------------------------------------- decode

def _codes(d, N, T, k, seed):
    rng = np.random.default_rng(seed)
    idx = rng.integers(0, N, size=(T, k)).astype(np.int32)
    idx[:, 0] = rng.integers(0, d, size=T)          # some basis slots
    idx[::5, -1] = -1                                # some padding
    return idx


def test_decode_matches_dense_product():
    d, N = 64, 1 << 12
    m = oracle.masks(d, 12)
    idx = _codes(d, N, 32, 16, 0)
    coef = np.random.default_rng(1).standard_normal(idx.shape)
    y = oracle.decode(d, m, idx, coef)
    Phi = dense_dictionary(d, m, N)
    want = np.stack([(coef[t][idx[t] >= 0, None] * Phi[idx[t][idx[t] >= 0]]).sum(0) for t in range(32)])
    assert np.allclose(y, want, atol=1e-13, rtol=0)


def test_decode_exact_linearity_dyadic():
    """decode(alpha a + beta b) == alpha decode(a) + beta decode(b), bit-exact for
    small-integer coefficients at d = 64 where 1/sqrt d = 1/8 is exact."""
    d, N = 64, 1 << 12
    m = oracle.masks(d, 12)
    idx = _codes(d, N, 16, 16, 2)
    rng = np.random.default_rng(3)
    a = rng.integers(-8, 9, idx.shape).astype(np.float64)
    b = rng.integers(-8, 9, idx.shape).astype(np.float64)
    lhs = oracle.decode(d, m, idx, 3 * a - 5 * b)
    rhs = 3 * oracle.decode(d, m, idx, a) - 5 * oracle.decode(d, m, idx, b)
    assert np.array_equal(lhs, rhs)


def test_decode_one_hot_is_the_direction():
    d = 64
    m = oracle.masks(d, 12)
    idx = np.array([[1000, -1]], np.int32)
    y = oracle.decode(d, m, idx, np.array([[1.0, 7.0]]))
    assert set(np.unique(y).tolist()) == {0.125, -0.125}


def test_decode_bwd_autograd_and_adjoint():
    """float64 autograd through a dense Phi_S: with coef = Phi_S x and
    y = Phi_S^T coef, the VJP for upstream g is grad_coef = Phi_S g and
    grad_x = Phi_S^T grad_coef (straight-through in the indices)."""
    d, N, T, k = 64, 1 << 12, 8, 16
    m = oracle.masks(d, 12)
    idx = _codes(d, N, T, k, 4)
    g = np.random.default_rng(5).standard_normal((T, d))
    gc, gx = oracle.decode_bwd(d, m, idx, g)
    Phi = torch.from_numpy(dense_dictionary(d, m, N))
    for t in range(T):
        live = idx[t] >= 0
        PhiS = Phi[torch.from_numpy(idx[t][live].astype(np.int64))]
        coef = torch.zeros(int(live.sum()), dtype=torch.float64, requires_grad=True)
        y = coef @ PhiS
        (gcoef,) = torch.autograd.grad(y, coef, torch.from_numpy(g[t]))
        assert np.allclose(gc[t][live], gcoef.numpy(), atol=1e-13)
        assert (gc[t][~live] == 0).all()
        x = torch.zeros(d, dtype=torch.float64, requires_grad=True)
        yx = (PhiS @ x) @ PhiS
        (gxx,) = torch.autograd.grad(yx, x, torch.from_numpy(g[t]))
        assert np.allclose(gx[t], gxx.numpy(), atol=1e-12)
    # adjoint: <decode(idx, a), g> == <a, grad_coef(idx, g)>
    a = np.random.default_rng(6).standard_normal((T, k))
    a[idx < 0] = 0
    y = oracle.decode(d, m, idx, a)
    assert abs((y * g).sum() - (a * gc).sum()) < 1e-10
    assert np.allclose(gx, oracle.decode(d, m, idx, gc), atol=1e-12)
