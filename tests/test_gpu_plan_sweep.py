"""GPU parity over a seeded sweep of hierarchies: dimensions with and without
ragged chunks, 2 to 5 levels, 16 to 256 children per parent, small and large
beams, fp32 and bf16, each against the oracle (encode, encode on
standardized scores with random statistics; decode and backward on the
oracle's codes).  The plans are drawn once from a fixed seed
(`sweep_plans`), so every run checks the same cases; a plan the library
declares unsupported is skipped with its reason."""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2607_20652_amd import binding as dpb
from paper_2607_20652_amd import inputs
from parity_util import TOL_BF16, TOL_F32, compare_dense, compare_encode, random_std_state, EncodeCheck

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def sweep_plans(n_plans=40, seed=2607):
    """(d, level bits, branchings, active, dtype, T) per case."""
    rng = np.random.default_rng(seed)
    dims = [64, 96, 200, 256, 384, 520, 768, 1000, 1024, 1536, 2048]
    out = []
    while len(out) < n_plans:
        d = int(rng.choice(dims))
        n0 = int(np.ceil(np.log2(d)))
        L = int(rng.integers(2, 6))
        nb, dl, K = [n0], [0], [int(rng.choice([2, 4, 8, 16]))]
        for _ in range(1, L):
            step = int(rng.integers(2, 6))
            if nb[-1] + step > 24:
                break
            nb.append(nb[-1] + step)
            room = (1 << nb[-1]) - (1 << nb[-2])
            delta = int(min(room, rng.choice([16, 32, 64, 128, 256])))
            dl.append(delta)
            K.append(int(min(K[-1] * delta, rng.choice([4, 8, 16, 32, 64]))))
        if len(nb) < 2:
            continue
        dtype = "f32" if rng.random() < 0.3 else "bf16"
        T = int(rng.integers(1, 120))
        out.append((d, nb, dl, K, dtype, T))
    return out


CASES = sweep_plans()


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    dpb.load()


@pytest.mark.parametrize("case", range(len(CASES)))
def test_plan_sweep(case):
    d, nb, dl, K, dt, T = CASES[case]
    say(f"[sweep {case}] d={d} n={nb} delta={dl} K={K} {dt} T={T}")
    try:
        plan = dpb.Plan(d, seed=0, level_bits=nb, branchings=dl, active=K)
    except dpb.DPBError as e:
        pytest.skip(f"unsupported plan: {e}")
    m = oracle.masks(d, nb[-1])
    gens = oracle.generators(nb, dl, 0)
    x = inputs.normal((T, d), 7000 + case, dt)
    xd = x.double().numpy()
    try:
        idx, coef = dpb.encode(plan, x.to(DEV))
    except dpb.DPBError as e:
        pytest.skip(f"unsupported encode: {e}")
    torch.cuda.synchronize()
    oi, oc, om, oo = oracle.encode(d, m, nb, K, dl, gens, xd)
    st = compare_encode(K, idx.cpu().numpy(), coef.cpu().numpy(), oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(d, m, gens, xd))
    say(f"  encode {st}")
    assert st["exempt_tokens"] <= max(2, 0.05 * T)

    # standardized scores (§2.2 "Score Standardization") with random statistics
    mu, _, r = random_std_state(1 << nb[-1], 7200 + case)
    stats = torch.from_numpy(np.stack([mu, r], axis=1)).contiguous().to(DEV)
    try:
        sidx, scoef = dpb.encode(plan, x.to(DEV), stats=stats)
    except dpb.DPBError as e:
        say(f"  standardized encode unsupported: {e}")
    else:
        torch.cuda.synchronize()
        si, sc, sm, so = oracle.encode_std(d, m, nb, K, dl, gens, xd, mu, r)
        st2 = compare_encode(K, sidx.cpu().numpy(), scoef.cpu().numpy(), si, sc, sm, so, TOL_F32,
                             ctx=EncodeCheck(d, m, gens, xd, mu, r))
        say(f"  encode std {st2}")
        assert st2["exempt_tokens"] <= max(2, 0.05 * T)

    tdt = torch.float32 if dt == "f32" else torch.bfloat16
    tol = TOL_F32 if dt == "f32" else TOL_BF16
    oc32 = oc.astype(np.float32)
    it = torch.from_numpy(oi).to(DEV)
    y = dpb.decode(plan, it, torch.from_numpy(oc32).to(DEV), tdt)
    g = inputs.normal((T, d), 7100 + case, dt)
    gc, gx = dpb.decode_bwd(plan, it, g.to(DEV))
    torch.cuda.synchronize()
    ey = compare_dense(y.float().cpu().numpy(), oracle.decode(d, m, oi, oc32.astype(np.float64)), tol)
    rgc, rgx = oracle.decode_bwd(d, m, oi, g.double().numpy())
    e1 = compare_dense(gc.cpu().numpy(), rgc, TOL_F32)
    e2 = compare_dense(gx.float().cpu().numpy(), rgx, tol)
    say(f"  y err {ey:.3g}  grad_coef err {e1:.3g}  grad_x err {e2:.3g}")
