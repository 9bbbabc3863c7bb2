"""CPU tests of the encode comparison rules used by the GPU parity tests:
an oracle code passes against itself, also when every hashed level is
treated as a near-tie (then each level is rescored from the code's own
parents), and planted mistakes in a copy of it are caught."""
import numpy as np
import pytest

import oracle
from paper_2607_20652_amd import inputs
from parity_util import TOL_F32, EncodeCheck, compare_encode


@pytest.fixture(scope="module")
def case():
    w = inputs.workload("gpt2")
    nb, dl, K = oracle.hierarchy(w.d, w.n, w.levels, w.branching, w.beam, w.k)
    m, g = oracle.masks(w.d, w.n), oracle.generators(nb, dl, 0)
    x = inputs.activations("gpt2", 24).double().numpy()
    oi, oc, om, oo = oracle.encode(w.d, m, nb, K, dl, g, x)
    return K, oi, oc, om, oo, EncodeCheck(w.d, m, g, x)


def run(case, idx, coef, all_near_ties):
    K, oi, oc, om, oo, ctx = case
    margin = np.zeros_like(om) if all_near_ties else om
    return compare_encode(K, idx, coef, oi, oc, margin, oo, TOL_F32, ctx)


@pytest.mark.parametrize("all_near_ties", [False, True])
def test_oracle_code_passes_against_itself(case, all_near_ties):
    K, oi, oc = case[0], case[1], case[2]
    st = run(case, oi.copy(), oc.copy(), all_near_ties)
    if all_near_ties:
        assert st["rescored_levels"] == oi.shape[0] * (len(K) - 1)


def _mutated(case, fn):
    oi, oc = case[1].copy(), case[2].copy()
    fn(oi, oc)
    return oi, oc


@pytest.mark.parametrize("all_near_ties", [False, True])
@pytest.mark.parametrize("mistake", ["foreign_index", "weak_candidate", "coef", "coef_row_scale", "order", "repeat",
                                     "padding"])
def test_planted_mistakes_are_caught(case, all_near_ties, mistake):
    K, _, _, _, _, ctx = case
    s1 = K[0]                     # first slot of level 1
    sL = sum(K[:-1])              # first slot of the last level
    t = 3

    def plant(oi, oc):
        if mistake == "foreign_index":      # an index no parent reaches
            oi[t, sL + 5] = (1 << 16) - 1 if (1 << 16) - 1 not in oi[t] else (1 << 16) - 2
        elif mistake == "weak_candidate":   # the last slot replaced by the weakest candidate
            par = oi[t, sum(K[:-2]):sL].astype(np.int64)
            cands = np.unique((par[:, None] ^ ctx.gens[len(K) - 1].astype(np.int64)[None, :]).reshape(-1))
            s = ctx.scores(t, cands)
            weak = cands[np.argmin(np.abs(s))]
            oi[t, sL + K[-1] - 1] = weak
            oc[t, sL + K[-1] - 1] = s[np.argmin(np.abs(s))]
        elif mistake == "coef":
            oc[t, s1 + 2] *= 1.0 + 1e-4
        elif mistake == "coef_row_scale":   # the weakest slot moved by 1e-4 of its level row's rms, toward 0
            row = oc[t, sL:sL + K[-1]]
            shift = 1e-4 * np.sqrt(np.mean(row * row))
            oc[t, sL + K[-1] - 1] -= np.sign(oc[t, sL + K[-1] - 1]) * shift
        elif mistake == "order":
            oi[t, [s1, s1 + 1]] = oi[t, [s1 + 1, s1]]
            oc[t, [s1, s1 + 1]] = oc[t, [s1 + 1, s1]]
        elif mistake == "repeat":
            oi[t, sL + 1] = oi[t, sL]
            oc[t, sL + 1] = oc[t, sL]
        elif mistake == "padding":
            oi[t, sL + 7] = -1
            oc[t, sL + 7] = 0.0

    oi, oc = _mutated(case, plant)
    with pytest.raises(AssertionError):
        run(case, oi, oc, all_near_ties)
