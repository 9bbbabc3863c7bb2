"""GPU parity of score standardization (§2.2 "Score Standardization")
through the C ABI: the standardized encoder, the EMA update of the
statistics, the backward with standardized coefficients, and the DPB layer
that updates its statistics after each training backward.

The encoder is compared with the rules of parity_util (level 0 exact: both
sides take z = (x - mu) r in fp32; near-ties exempt above); the statistics
within 1e-5 relative plus 1e-5 absolute (fp32 EMA arithmetic on fp64
moments of fp32 raw scores of order 1; see the update test).
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2607_20652_amd import autograd as dpb_autograd
from paper_2607_20652_amd import binding as dpb
from paper_2607_20652_amd import inputs
from parity_util import TOL_BF16, TOL_F32, compare_dense, compare_encode, random_std_state, EncodeCheck

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
_PLANS = {}


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    dpb.load()


def plan_for(name):
    if name not in _PLANS:
        w = inputs.workload(name)
        _PLANS[name] = dpb.Plan(w.d, w.n, w.levels, w.branching, w.beam, w.k, 0)
    return _PLANS[name]


def setup(name):
    w = inputs.workload(name)
    nb, dl, K = oracle.hierarchy(w.d, w.n, w.levels, w.branching, w.beam, w.k)
    return w, nb, dl, K, oracle.masks(w.d, w.n), oracle.generators(nb, dl, 0)


def random_state(N, seed, scale=1.0):
    return random_std_state(N, seed, scale)


def device_stats(mu, r):
    return torch.from_numpy(np.stack([mu, r], axis=1)).contiguous().to(DEV)


@pytest.mark.parametrize("name,T", [("tiny", 256), ("train", 300)])
def test_identity_state_equals_plain_encoder(name, T):
    say(f"[std identity] {name} T={T}")
    plan = plan_for(name)
    x = inputs.activations(name, T).to(DEV)
    stats, _ = dpb.std_state(plan)
    i1, c1 = dpb.encode(plan, x)
    i2, c2 = dpb.encode_std(plan, x, stats)
    torch.cuda.synchronize()
    assert torch.equal(i1, i2) and torch.equal(c1, c2)


@pytest.mark.parametrize("name,T,f32", [("tiny", 256, False), ("gpt2", 500, False), ("gpt2", 200, True),
                                        ("train", 400, False), ("very_wide", 120, False)])
def test_encode_std_matches_oracle(name, T, f32):
    say(f"[encode std] {name} T={T} f32={f32}")
    plan = plan_for(name)
    w, nb, dl, K, m, gens = setup(name)
    x = inputs.normal((T, w.d), 400 + w.index) if f32 else inputs.activations(name, T)
    mu, _, r = random_state(1 << w.n, 11 + w.index)
    idx, coef = dpb.encode_std(plan, x.to(DEV), device_stats(mu, r))
    torch.cuda.synchronize()
    oi, oc, om, oo = oracle.encode_std(w.d, m, nb, K, dl, gens, x.double().numpy(), mu, r)
    st = compare_encode(K, idx.cpu().numpy(), coef.cpu().numpy(), oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(w.d, m, gens, x.double().numpy(), mu, r))
    say(f"  {st}")
    assert st["exempt_tokens"] <= max(2, 0.02 * T)


def test_encode_std_full_size_sampled():
    name = "train"
    w, nb, dl, K, m, gens = setup(name)
    say(f"[encode std full] {name} T={w.tokens}")
    plan = plan_for(name)
    x = inputs.activations(name)
    mu, _, r = random_state(1 << w.n, 21)
    idx, coef = dpb.encode_std(plan, x.to(DEV), device_stats(mu, r))
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(64), np.random.default_rng(2).choice(w.tokens, 128, replace=False),
                                     np.arange(w.tokens - 64, w.tokens)]))
    oi, oc, om, oo = oracle.encode_std(w.d, m, nb, K, dl, gens, x[rows].double().numpy(), mu, r)
    st = compare_encode(K, idx.cpu().numpy()[rows], coef.cpu().numpy()[rows], oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(w.d, m, gens, x[rows].double().numpy(), mu, r))
    say(f"  {st}")
    assert st["exempt_tokens"] <= max(2, 0.02 * len(rows))


@pytest.mark.parametrize("name,T,beta", [("tiny", 300, 0.1), ("tiny", 40, 1.0), ("gpt2", 1000, 0.05),
                                         ("train", 2048, 0.02), ("very_wide", 90, 0.3)])
def test_std_update_matches_oracle(name, T, beta):
    say(f"[std update] {name} T={T} beta={beta}")
    plan = plan_for(name)
    w, nb, dl, K, m, gens = setup(name)
    N = 1 << w.n
    mu, m2, r = random_state(N, 31 + w.index)
    stats = device_stats(mu, r)
    m2d = torch.from_numpy(m2).to(DEV)
    x = inputs.activations(name, T)
    idx, _ = dpb.encode_std(plan, x.to(DEV), stats)
    before = stats.clone()
    dpb.std_update(plan, x.to(DEV), idx, stats, m2d, beta, 1e-6)
    torch.cuda.synchronize()
    rmu, rm2 = oracle.std_update(w.d, m, nb, K, dl, gens, x.double().numpy(), idx.cpu().numpy(),
                                  mu.astype(np.float64), m2.astype(np.float64), beta)
    gs, gv = stats.cpu().numpy(), m2d.cpu().numpy()
    touched = (rmu != mu.astype(np.float64)) | (rm2 != m2.astype(np.float64))
    say(f"  touched {int(touched.sum())} of {N}")
    assert np.array_equal(gs[~touched], before.cpu().numpy()[~touched])
    assert np.array_equal(gv[~touched], m2[~touched])
    # raw scores here are O(1) (unit-norm directions, unit-variance inputs):
    # fp32 accumulation and the fp32 state update move mean and second moment
    # by ~1e-6 absolutely, hence the absolute part of the bound
    assert np.allclose(gs[touched, 0], rmu[touched], rtol=1e-5, atol=1e-5)
    assert np.allclose(gv[touched], rm2[touched], rtol=1e-5, atol=1e-5)
    # r is the one the GPU's own fp32 (mu, m2) imply (fp32 subtraction m2 - mu^2)
    rr = oracle.std_r(gs[touched, 0].astype(np.float64), gv[touched].astype(np.float64), 1e-6)
    assert np.allclose(gs[touched, 1], rr, rtol=2e-6, atol=0)
    # and the oracle's own state's r where the variance is not a small
    # difference of the two moments (there fp32 rounding of m2 and mu^2
    # dominates it: e.g. a single sample with beta = 1 has variance exactly 0)
    well = touched & (rm2 - rmu ** 2 > 1e-2 * rm2)
    ro = oracle.std_r(rmu[well], rm2[well], 1e-6)
    assert np.allclose(gs[well, 1], ro, rtol=1e-4, atol=0)
    if beta < 1.0:
        assert well.sum() > 0.9 * touched.sum()


@pytest.mark.parametrize("name,T", [("tiny", 77), ("train", 500)])
def test_decode_bwd_with_stats(name, T):
    say(f"[bwd std] {name} T={T}")
    plan = plan_for(name)
    w, nb, dl, K, m, gens = setup(name)
    mu, _, r = random_state(1 << w.n, 41)
    stats = device_stats(mu, r)
    x = inputs.activations(name, T).to(DEV)
    idx, _ = dpb.encode_std(plan, x, stats)
    g = inputs.upstream_grad(name, T).to(DEV)
    agc = inputs.normal((T, plan.k_tot), 43).to(DEV)
    gc, gx = dpb.decode_bwd_ex(plan, idx, g, add_grad_coef=agc, stats=stats)
    torch.cuda.synchronize()
    ii = idx.cpu().numpy()
    rgc, _ = oracle.decode_bwd(w.d, m, ii, g.double().cpu().numpy())
    rgc = rgc + agc.double().cpu().numpy()
    rs = np.where(ii >= 0, r[np.maximum(ii, 0)], 0.0)
    rgx = oracle.decode(w.d, m, ii, rgc * rs)
    compare_dense(gc.cpu().numpy(), rgc, TOL_F32)
    compare_dense(gx.float().cpu().numpy(), rgx, TOL_F32 if w.dtype == "f32" else TOL_BF16)


@pytest.mark.parametrize("name,T", [("tiny", 200), ("train", 512)])
def test_standardized_layer_matches_oracle_and_updates(name, T):
    say(f"[std layer] {name} T={T}")
    plan = plan_for(name)
    w, nb, dl, K, m, gens = setup(name)
    std = dpb_autograd.Standardizer(plan, momentum=0.1, eps=1e-6)
    mu, m2, r = random_state(1 << w.n, 51)
    std.stats.copy_(device_stats(mu, r))
    std.m2.copy_(torch.from_numpy(m2))
    x = inputs.activations(name, T).to(DEV).requires_grad_(True)
    gy = inputs.upstream_grad(name, T).to(DEV)
    y, lv = dpb_autograd.dpb_layer(x, plan, True, 2, std)
    idx, coef = dpb.encode_std(plan, x.detach(), device_stats(mu, r))
    torch.autograd.backward([y, lv], [gy, torch.tensor(0.5, device=DEV)])
    torch.cuda.synchronize()
    ii, cc = idx.cpu().numpy(), coef.cpu().numpy().astype(np.float64)
    xd = x.detach().double().cpu().numpy()
    ry, _ = oracle.normalize(oracle.decode(w.d, m, ii, cc), xd)
    compare_dense(y.detach().float().cpu().numpy(), ry, TOL_F32 if w.dtype == "f32" else TOL_BF16)
    rs = np.where(ii >= 0, r[np.maximum(ii, 0)], 0.0)
    _, rgx = oracle.layer_backward(w.d, m, ii, cc, xd, gy.double().cpu().numpy(), 0.5, 2, True, r_slot=rs)
    compare_dense(x.grad.float().cpu().numpy(), rgx, TOL_F32 if w.dtype == "f32" else TOL_BF16)
    # the training backward applied the EMA update of this batch
    rmu, rm2 = oracle.std_update(w.d, m, nb, K, dl, gens, xd, ii, mu.astype(np.float64), m2.astype(np.float64),
                                  0.1)
    gs = std.stats.cpu().numpy()
    assert np.allclose(gs[:, 0], rmu, rtol=1e-5, atol=1e-5)
    assert np.allclose(std.m2.cpu().numpy(), rm2, rtol=1e-5, atol=1e-5)
