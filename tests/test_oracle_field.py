"""Pins for the oracle's finite-field layer (App. A.2, A.4).

Each test checks the oracle against something other than itself: the paper's
printed moduli, Gauss's count of irreducible polynomials, the field axioms
(exhaustively at small t) and the properties of the trace proved in App. A.2.
"""
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")))


def _mul_table(t, poly):
    n = 1 << t
    return np.array([[oracle.gf_mul(a, b, t, poly) for b in range(n)] for a in range(n)], dtype=np.int64)


def test_paper_moduli():
    """The modulus rule reproduces z^10+z^3+1 and z^11+z^2+1 (App. A.4)."""
    for t in ("10", "11"):
        want = sum(1 << e for e in GOLDEN["irreducible_polys"][t]["terms"])
        assert want == GOLDEN["irreducible_polys"][t]["value"]
        assert oracle.pick_poly(int(t)) == want


def _moebius(n):
    res, p, m = 1, 2, n
    while p * p <= m:
        if m % p == 0:
            m //= p
            if m % p == 0:
                return 0
            res = -res
        p += 1
    if m > 1:
        res = -res
    return res


@pytest.mark.parametrize("t", range(1, 11))
def test_irreducible_count_matches_gauss_formula(t):
    """# irreducible binary polynomials of degree t = (1/t) sum_{e|t} mu(e) 2^{t/e}."""
    want = sum(_moebius(e) * 2 ** (t // e) for e in range(1, t + 1) if t % e == 0) // t
    got = sum(oracle.poly_irreducible(f) for f in range(1 << t, 1 << (t + 1)))
    assert got == want


def test_field_axioms_exhaustive_t6():
    """z^6+z+1 gives a field: commutative, associative, distributive, inverses."""
    t, poly = 6, oracle.pick_poly(6)
    assert poly == 0b1000011
    M = _mul_table(t, poly)
    n = 1 << t
    a = np.arange(n)
    assert (M == M.T).all()
    assert (M[1] == a).all() and (M[0] == 0).all()
    # associativity (a b) c == a (b c) over all triples
    assert (M[M[:, :, None], a[None, None, :]] == M[a[:, None, None], M[None, :, :]]).all()
    # distributivity a (b + c) == a b + a c, + is XOR
    lhs = M[a[:, None, None], (a[None, :, None] ^ a[None, None, :])]
    rhs = M[:, :, None] ^ M[:, None, :]
    assert (lhs == rhs).all()
    # every nonzero row is a permutation of the nonzero elements (no zero divisors)
    for x in range(1, n):
        assert sorted(M[x, 1:].tolist()) == list(range(1, n))


def test_reducible_modulus_has_zero_divisors():
    """Control: the same multiplication with a reducible modulus is not a field."""
    t, poly = 6, 0b1000001  # z^6 + 1 = (z+1)^2 (z^2+z+1)^2, reducible
    assert not oracle.poly_irreducible(poly)
    M = _mul_table(t, poly)
    assert (M[1:, 1:] == 0).any()


@pytest.mark.parametrize("t", [6, 10, 11])
def test_inverse_exhaustive(t):
    """xi * xi^{-1} = 1 for every nonzero xi; the inverse is an involution; 0^{-1} = 0."""
    poly = oracle.pick_poly(t)
    assert oracle.gf_inv(0, t, poly) == 0
    for x in range(1, 1 << t):
        inv = oracle.gf_inv(x, t, poly)
        assert oracle.gf_mul(x, inv, t, poly) == 1
        assert oracle.gf_inv(inv, t, poly) == x


@pytest.mark.parametrize("t", [6, 10])
def test_trace_lemma(t):
    """Properties of the trace (App. A.2): values in {0,1}, additive, not identically 0,
    and balanced over the field (the balanced-parities lemma with alpha = 1)."""
    poly = oracle.pick_poly(t)
    n = 1 << t
    tr = np.array([oracle.gf_trace(y, t, poly) for y in range(n)])
    assert set(tr.tolist()) <= {0, 1}
    assert tr[0] == 0 and tr.sum() == n // 2
    rng = np.random.default_rng(t)
    for y, z in rng.integers(0, n, size=(500, 2)):
        assert tr[y ^ z] == tr[y] ^ tr[z]
    # Tr(y^2) = Tr(y): squaring permutes the terms of the trace sum
    for y in range(n):
        assert tr[oracle.gf_mul(y, y, t, poly)] == tr[y]


@pytest.mark.parametrize("t", [6, 10])
def test_trace_as_parity(t):
    """Tr(a xi) = <coord xi, tau(a)> with tau(a)_q = Tr(a z^q); tau is a bijection
    (App. A.4, trace-as-parity equation)."""
    poly = oracle.pick_poly(t)
    n = 1 << t
    taus = []
    rng = np.random.default_rng(1)
    a_vals = range(n) if t <= 6 else rng.integers(0, n, size=64)
    for a in a_vals:
        tau = 0
        for q in range(t):
            tau |= oracle.gf_trace(oracle.gf_mul(int(a), 1 << q, t, poly), t, poly) << q
        taus.append(tau)
        for xi in (range(n) if t <= 6 else rng.integers(0, n, size=128)):
            direct = oracle.gf_trace(oracle.gf_mul(int(a), int(xi), t, poly), t, poly)
            assert direct == bin(int(xi) & tau).count("1") % 2
    if t <= 6:
        assert sorted(taus) == list(range(n))


def test_z_is_primitive_for_t10():
    """Reading for d = 768: z has order 2^10 - 1 under z^10+z^3+1, so the
    coordinates z^0..z^766 are distinct (parity unpinned against the paper)."""
    poly = oracle.pick_poly(10)
    assert oracle.gf_order(2, 10, poly) == 1023
    assert oracle.primitive_element(10, poly) == 2
