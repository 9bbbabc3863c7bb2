"""Pins for the oracle's plan constants that rest on readings of the paper:
the generator sampling (§2.2 fixes only that a level's generators are
distinct values of that level's index range; the sampling rule is reading R6)
and the mapping from configuration terms to per-level sizes (reading R12, the
table of the hot-path scope), plus the precision reading of standardized
level-0 scores (R20).

What is pinned against something other than the oracle itself:
  * the SplitMix64 stream against its published reference outputs
    (tests/golden/splitmix64_reference.json);
  * every level's generators against the range and distinctness §2.2 asks
    for, including the full-set corner case;
  * the level bit widths against the values the scope table lists for the
    GPT-2, wide and very wide configurations (where the rounding of
    l (n - n_0) / (L - 1) matters);
  * fp32 level-0 z against fp64 z: the same selection wherever the fp64
    margin is not a near-tie.
"""
import json
import os

import numpy as np
import pytest

import oracle
from paper_2607_20652_amd import inputs

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
GAMMA = 0x9E3779B97F4A7C15


def test_splitmix64_matches_published_reference_outputs():
    ref = json.load(open(os.path.join(GOLDEN, "splitmix64_reference.json")))
    got = oracle.splitmix64(ref["seed"], len(ref["outputs"]))
    assert got == [int(v) for v in ref["outputs"]]


@pytest.mark.parametrize("nbits,delta,seed", [
    ([6, 9, 12], [0, 16, 16], 0),
    ([10, 12, 14, 16], [0, 16, 16, 16], 0),
    ([10, 12, 15, 17, 20], [0, 16, 16, 16, 16], 12345),
    ([10, 12, 15, 18, 21, 24], [0, 16, 16, 16, 16, 16], 7),
    ([10, 15, 17], [0, 256, 256], 0),
    ([11, 15], [0, 256], 3),
    ([6, 7, 9], [0, 64, 300], 99),          # level 1 nearly, level 2 heavily subsampled
])
def test_generators_are_distinct_values_of_their_level(nbits, delta, seed):
    gens = oracle.generators(nbits, delta, seed)
    for l in range(1, len(nbits)):
        g = gens[l].astype(np.int64)
        assert g.shape == (delta[l],)
        assert np.unique(g).size == delta[l]
        assert g.min() >= 1 << nbits[l - 1] and g.max() < 1 << nbits[l]
        # a generator with a set bit at or above n_{l-1} moves a parent of the
        # level below into level l: p XOR g lies in [2^{n_{l-1}}, 2^{n_l})
        p = np.arange(0, 1 << nbits[l - 1], max(1, (1 << nbits[l - 1]) // 64))
        c = p[:, None] ^ g[None, :]
        assert (c >= 1 << nbits[l - 1]).all() and (c < 1 << nbits[l]).all()


def test_full_generator_set_is_the_whole_level():
    nbits = [6, 9, 12]
    delta = [0, (1 << 9) - (1 << 6), (1 << 12) - (1 << 9)]
    gens = oracle.generators(nbits, delta, 5)
    for l in (1, 2):
        assert np.array_equal(np.sort(gens[l]), np.arange(1 << nbits[l - 1], 1 << nbits[l], dtype=np.uint32))


def test_generators_follow_the_splitmix64_stream_of_their_level():
    """Consistency of the sampler with the pinned stream (R6): level l takes the
    low n_l bits of the stream from state seed ^ (l * gamma), in order,
    skipping values below 2^{n_{l-1}} and repeats.  Different seeds and levels
    give different sets."""
    nbits, delta, seed = [10, 12, 15, 17, 20], [0, 16, 16, 16, 16], 12345
    gens = oracle.generators(nbits, delta, seed)
    for l in range(1, len(nbits)):
        stream = oracle.splitmix64(seed ^ ((l * GAMMA) & (2**64 - 1)), 4096)
        want = []
        for v in stream:
            v &= (1 << nbits[l]) - 1
            if v >= 1 << nbits[l - 1] and v not in want:
                want.append(v)
            if len(want) == delta[l]:
                break
        assert [int(v) for v in gens[l]] == want
    other = oracle.generators(nbits, delta, seed + 1)
    assert not any(np.array_equal(other[l], gens[l]) for l in range(1, len(nbits)))


def test_generators_are_spread_over_their_level():
    """A large draw covers the level's range evenly (chi-square over 16 bins):
    a sampler that took the wrong bits of the stream, or folded values into
    part of the range, fails this."""
    nbits, delta = [8, 16], [0, 8000]
    g = oracle.generators(nbits, delta, 11)[1].astype(np.int64) - (1 << 8)
    span = (1 << 16) - (1 << 8)
    counts = np.bincount(g * 16 // span, minlength=16)
    exp = delta[1] / 16
    chi2 = float(((counts - exp) ** 2 / exp).sum())
    assert chi2 < 40.0   # 15 degrees of freedom: p ~ 5e-4


# level bits, branching and active counts of the scope table (§8.0) for the
# configurations where floor(l (n - n0) / (L - 1)) is not exact
SCOPE_TABLE = {
    "tiny": ([6, 9, 12], [0, 16, 16], [4, 4, 8]),
    "gpt2": ([10, 12, 14, 16], [0, 16, 16, 16], [8, 8, 8, 32]),
    "wide": ([10, 12, 15, 17, 20], [0, 16, 16, 16, 16], [8, 8, 8, 8, 64]),
    "very_wide": ([10, 12, 15, 18, 21, 24], [0, 16, 16, 16, 16, 16], [16, 16, 16, 16, 16, 64]),
}


@pytest.mark.parametrize("name", list(SCOPE_TABLE))
def test_hierarchy_matches_scope_table(name):
    w = inputs.workload(name)
    nb, dl, K = oracle.hierarchy(w.d, w.n, w.levels, w.branching, w.beam, w.k)
    assert (nb, dl, K) == SCOPE_TABLE[name]
    assert sum(K) == {"tiny": 16, "gpt2": 56, "wide": 96, "very_wide": 144}[name]


def _level0_fp64(x, mu, r, K):
    """Top-K of |z| with z = (x - mu) r in fp64, ties to the lower index, and
    the fp64 boundary margin (|z|_(K) - |z|_(K+1)) / |z|_(K) per token."""
    z = (x - mu.astype(np.float64)[None, :]) * r.astype(np.float64)[None, :]
    sel, margin = [], []
    for row in z:
        order = np.lexsort((np.arange(row.size), -np.abs(row)))
        sel.append(np.sort(order[:K]))
        a, b = abs(row[order[K - 1]]), abs(row[order[K]])
        margin.append((a - b) / a if a > 0 else 0.0)
    return np.array(sel), np.array(margin)


@pytest.mark.parametrize("name", ["tiny", "gpt2"])
def test_level0_standardized_selection_in_fp32_equals_fp64_off_near_ties(name):
    """Reading R20 takes level-0 z in fp32 (the precision the kernel takes it
    in).  That can change the selected set only where the fp64 selection has
    a near-tie at its boundary: elsewhere the two precisions select the same
    features."""
    w = inputs.workload(name)
    nb, dl, K = oracle.hierarchy(w.d, w.n, w.levels, w.branching, w.beam, w.k)
    m, g = oracle.masks(w.d, w.n), oracle.generators(nb, dl, 0)
    T = 400 if name == "tiny" else 120
    x = inputs.activations(name, T).double().numpy()
    rng = np.random.default_rng(5)
    N = 1 << w.n
    mu = (0.3 * rng.standard_normal(N)).astype(np.float32)
    r = rng.uniform(0.5, 2.0, N).astype(np.float32)
    idx, _, _, _ = oracle.encode_std(w.d, m, nb, K, dl, g, x, mu, r)
    sel64, margin = _level0_fp64(x, mu[: w.d], r[: w.d], K[0])
    ok = margin >= 1e-6
    assert ok.sum() > 0.9 * T
    got = np.sort(idx[:, : K[0]], axis=1)
    assert np.array_equal(got[ok], sel64[ok])
