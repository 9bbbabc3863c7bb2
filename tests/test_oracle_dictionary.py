"""Pins for the oracle's dictionary: seed matrix M, directions, coherence.

Against: the Kloosterman codeword definition computed with field arithmetic
(App. A.3), the exact coherence spectrum of the proof of the coherence theorem
(Cases 1-3) and of the attribution remark after the Weil bound, the paper's
printed bounds, and the exact-value facts of §2.1.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")))


def _tau(a, t, poly):
    return sum(oracle.gf_trace(oracle.gf_mul(a, 1 << q, t, poly), t, poly) << q for q in range(t))


@pytest.mark.parametrize("t,exhaustive", [(6, True), (10, False)])
def test_masks_generate_kloosterman_code(t, exhaustive):
    """Index u = (tau(a), tau(b)) gives the sign (-1)^{Tr(a xi + b xi^-1)} at every
    coordinate xi (App. A.3 Kloosterman-codeword eq.; App. A.4 coordinate-from-mask eq.)."""
    d = 1 << t
    poly = oracle.pick_poly(t)
    m = oracle.masks(d, 2 * t)
    rng = np.random.default_rng(7)
    pairs = [(a, b) for a in range(d) for b in range(d)] if exhaustive else rng.integers(0, d, (40, 2))
    coords = range(d) if exhaustive else rng.integers(0, d, 64)
    for a, b in pairs:
        u = _tau(int(a), t, poly) | (_tau(int(b), t, poly) << t)
        for xi in coords:
            xi = int(xi)
            inv = oracle.gf_inv(xi, t, poly)
            want = oracle.gf_trace(oracle.gf_mul(int(a), xi, t, poly) ^ oracle.gf_mul(int(b), inv, t, poly), t, poly)
            assert bin(int(m[xi]) & u).count("1") % 2 == want


def test_seed_matrix_shape_d2048():
    """For d = 2048, M has 2048 rows and 22 columns (App. A.4)."""
    g = GOLDEN["seed_matrix_shape"]
    m = oracle.masks(g["d"], 22)
    assert m.shape[0] == g["rows"]
    assert int(m.max()).bit_length() == g["columns"]


def _spectrum(d, r):
    return oracle.walsh_spectrum(d, oracle.masks(d, r), r)


@pytest.mark.parametrize("t", [6, 8, 10])
def test_exact_coherence_spectrum(t):
    """Proof of the coherence theorem: S(u) = 0 when exactly one half of u is 0
    (Cases 2 and 3), S(0) = d, and otherwise S(u) - 1 is a Kloosterman sum whose
    values are exactly the integers = -1 (mod 4) in [-2 sqrt d, 2 sqrt d]."""
    d, r = 1 << t, 2 * t
    S = _spectrum(d, r).reshape(1 << t, 1 << t)  # [high half, low half]
    assert S[0, 0] == d
    assert (S[0, 1:] == 0).all() and (S[1:, 0] == 0).all()
    K = S[1:, 1:] - 1
    kv = GOLDEN["kloosterman_values"]
    lim = 2 * math.sqrt(d)
    want = {v for v in range(-int(lim) - 1, int(lim) + 2) if abs(v) <= lim and v % kv["congruence_mod"] == kv["residue"] % kv["congruence_mod"]}
    assert set(np.unique(K).tolist()) == want


@pytest.mark.parametrize("t", [6, 8, 10, 11])
def test_coherence_theorem_bound(t):
    """mu <= (1 + 2 sqrt d)/d over all hashed pairs; mu = 2/sqrt d exactly for even t."""
    d = 1 << t
    S = _spectrum(d, 2 * t)
    mu = np.abs(S[1:]).max() / d
    assert mu <= (1 + 2 * math.sqrt(d)) / d + 1e-15
    if t % 2 == 0:
        assert mu == 2 / math.sqrt(d)


def test_printed_bound_values():
    """The bound is 'approximately 0.06' at d = 1024 and '0.04' at d = 2048."""
    g = GOLDEN["coherence_bound"]
    for d, printed in g["printed"].items():
        d = int(d)
        assert abs((1 + 2 * math.sqrt(d)) / d - printed) <= g["printed_rounding"]


@pytest.mark.parametrize("d,r", [(64, 12), (768, 16), (768, 20), (1024, 24)])
def test_entries_and_norms(d, r):
    """Every hashed entry is +-1/sqrt d, every direction has unit norm, and a basis
    vector meets every hashed vector with inner product exactly 1/sqrt d in magnitude."""
    m = oracle.masks(d, r)
    rng = np.random.default_rng(d + r)
    mag = 1 / math.sqrt(d)
    for i in rng.integers(d, 1 << r, 24):
        v = oracle.phi(d, m, int(i))
        assert set(np.unique(v).tolist()) <= {mag, -mag}
        assert abs(np.dot(v, v) - 1) < 1e-12
        j = int(rng.integers(0, d))
        assert abs(abs(np.dot(v, oracle.phi(d, m, j))) - mag) < 1e-15
    for j in range(3):
        e = oracle.phi(d, m, j)
        assert e[j] == 1 and np.count_nonzero(e) == 1


def test_child_factorization_d64():
    """phi~_{p XOR g} = phi~_p (.) R(M g) (§2.2 factorization eq.) for sampled
    p, g over the full 12-bit index space at d = 64."""
    d, r = 64, 12
    m = oracle.masks(d, r)
    rng = np.random.default_rng(5)
    mag = 1 / math.sqrt(d)
    for p, g in rng.integers(d, 1 << r, (64, 2)):
        child = int(p) ^ int(g)
        if child < d:
            continue
        lhs = oracle.phi(d, m, child)
        gamma = np.where([bin(int(mm) & int(g)).count("1") % 2 for mm in m], -1.0, 1.0)
        assert np.array_equal(lhs, oracle.phi(d, m, int(p)) * gamma)
        assert np.all(np.abs(lhs) == mag)


def test_d768_reading_properties():
    """Reading for d = 768 (parity unpinned against the paper): rows are distinct
    field coordinates, and the measured coherence is recorded."""
    m = oracle.masks(768, 20)
    low = m & 0x3FF
    assert len(set(low.tolist())) == 768
    S = oracle.walsh_spectrum(768, m, 20)
    assert np.abs(S[1:]).max() == 102      # mu = 102/768 = 0.1328
    S16 = oracle.walsh_spectrum(768, m, 16)
    assert np.abs(S16[1:]).max() == 98     # mu = 98/768 = 0.1276


def test_r24_extension_reading():
    """Reading for n = 24 > 2t at d = 1024 (parity unpinned against the paper):
    the first 20 columns are the paper's; the measured coherence is recorded."""
    m24 = oracle.masks(1024, 24)
    m20 = oracle.masks(1024, 20)
    assert np.array_equal(m24 & 0xFFFFF, m20)
    S = oracle.walsh_spectrum(1024, m24, 24)
    assert np.abs(S[1:]).max() == 120      # mu = 120/1024
