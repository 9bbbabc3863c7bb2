"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Every input is seeded (paper_2607_20652_amd.inputs); decode and backward are
fed the oracle's own codes so that near-tie exemptions of the encoder never
leak into their checks.  Full-size workloads run on the GPU in the launch
configuration the benchmark times; the oracle checks a sample of rows.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2607_20652_amd import binding as dpb
from paper_2607_20652_amd import inputs
from parity_util import TOL_BF16, TOL_F32, compare_dense, compare_encode, EncodeCheck

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    dpb.load()


_PLANS = {}
_FULL = {}


def full_activations(name):
    if name not in _FULL:
        _FULL[name] = inputs.activations(name)
    return _FULL[name]


def plan_for(name, seed=0):
    key = (name, seed)
    if key not in _PLANS:
        w = inputs.workload(name)
        _PLANS[key] = dpb.Plan(w.d, w.n, w.levels, w.branching, w.beam, w.k, seed)
    return _PLANS[key]


def oracle_setup(name, seed=0):
    w = inputs.workload(name)
    nb, dl, K = oracle.hierarchy(w.d, w.n, w.levels, w.branching, w.beam, w.k)
    return w, nb, dl, K, oracle.masks(w.d, w.n), oracle.generators(nb, dl, seed)


def sample_rows(T, n, seed=0):
    if T <= n:
        return np.arange(T)
    rng = np.random.default_rng(seed)
    mid = rng.choice(np.arange(64, T - 64), size=n - 128, replace=False)
    return np.unique(np.concatenate([np.arange(64), mid, np.arange(T - 64, T)]))


# ---------------------------------------------------------------- encode

@pytest.mark.parametrize("name,T", [("tiny", 256), ("tiny", 37), ("gpt2", 1000), ("wide", 333),
                                    ("very_wide", 150)])
def test_encode_matches_oracle(name, T):
    say(f"[encode] {name} T={T}")
    plan = plan_for(name)
    w, nb, dl, K, m, gens = oracle_setup(name)
    x = inputs.activations(name, T)
    idx, coef = dpb.encode(plan, x.to(DEV))
    torch.cuda.synchronize()
    oi, oc, om, oo = oracle.encode(w.d, m, nb, K, dl, gens, x.double().numpy())
    st = compare_encode(K, idx.cpu().numpy(), coef.cpu().numpy(), oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(w.d, m, gens, x.double().numpy()))
    say(f"  {st}")
    assert st["exempt_tokens"] <= max(2, 0.02 * T)


@pytest.mark.parametrize("name,T", [("gpt2", 300), ("wide", 257), ("very_wide", 90)])
def test_encode_f32_input_matches_oracle(name, T):
    """fp32 activations at the bf16 workloads' shapes (the fp32 scoring path)."""
    say(f"[encode f32] {name} T={T}")
    plan = plan_for(name)
    w, nb, dl, K, m, gens = oracle_setup(name)
    x = inputs.normal((T, w.d), 300 + w.index)
    idx, coef = dpb.encode(plan, x.to(DEV))
    torch.cuda.synchronize()
    oi, oc, om, oo = oracle.encode(w.d, m, nb, K, dl, gens, x.double().numpy())
    st = compare_encode(K, idx.cpu().numpy(), coef.cpu().numpy(), oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(w.d, m, gens, x.double().numpy()))
    say(f"  {st}")
    assert st["exempt_tokens"] <= max(2, 0.02 * T)


@pytest.mark.parametrize("name,rows", [("gpt2", 384), ("wide", 256), ("very_wide", 160)])
def test_encode_full_size_sampled(name, rows):
    w = inputs.workload(name)
    say(f"[encode full] {name} T={w.tokens}")
    plan = plan_for(name)
    _, nb, dl, K, m, gens = oracle_setup(name)
    x = full_activations(name)
    idx, coef = dpb.encode(plan, x.to(DEV))
    torch.cuda.synchronize()
    r = sample_rows(w.tokens, rows, seed=w.index)
    oi, oc, om, oo = oracle.encode(w.d, m, nb, K, dl, gens, x[r].double().numpy())
    st = compare_encode(K, idx.cpu().numpy()[r], coef.cpu().numpy()[r], oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(w.d, m, gens, x[r].double().numpy()))
    say(f"  {st}")
    assert st["exempt_tokens"] <= max(2, 0.02 * len(r))
    # every emitted index is unique within its token and lies in its level
    ih = idx.cpu().numpy()
    s = np.sort(ih, axis=1)
    assert not np.any((s[:, 1:] == s[:, :-1]) & (s[:, 1:] >= 0))
    slot = 0
    for l, k in enumerate(K):
        lo = 0 if l == 0 else 1 << nb[l - 1]
        hi = w.d if l == 0 else 1 << nb[l]
        blk = ih[:, slot:slot + k]
        assert ((blk >= lo) & (blk < hi)).all()
        slot += k


def test_encode_exhaustive_generators_tiny():
    """Full generator sets: every parent reaches its whole next level, so the
    search prunes nothing and repeats each child once per parent (heavy dedup)."""
    say("[encode exhaustive] d=64 n=(6,8,10)")
    d, nb, K = 64, [6, 8, 10], [4, 4, 8]
    full = [np.arange(1 << nb[l - 1], 1 << nb[l], dtype=np.uint32) for l in (1, 2)]
    dl = [0, len(full[0]), len(full[1])]
    plan = dpb.Plan(d, level_bits=nb, branchings=dl, active=K, generators=np.concatenate(full).tolist())
    x = inputs.activations("tiny", 200)
    idx, coef = dpb.encode(plan, x.to(DEV))
    torch.cuda.synchronize()
    m = oracle.masks(d, nb[-1])
    oi, oc, om, oo = oracle.encode(d, m, nb, K, dl, [np.zeros(0, np.uint32)] + full, x.double().numpy())
    st = compare_encode(K, idx.cpu().numpy(), coef.cpu().numpy(), oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(d, m, [np.zeros(0, np.uint32)] + full, x.double().numpy()))
    say(f"  {st}")


# Narrow-encoder plans with 32 and 64 children per parent: 8 or 16 keys per
# lane (two or four generator tiles) in the threshold selection of the beam
# levels, whose per-lane counts then need 4 or 5 bits.  "k2" keeps 2 level-0
# parents and 16 of their 64 children, so fewer lanes than K_1 hold keys: the
# threshold is 1 and every live lane counts all 8 of its keys.
NARROW_BRANCHY = {
    "k2": dict(d=2048, level_bits=(11, 14, 17), branchings=(0, 32, 32), active=(2, 16, 24)),
    "b32": dict(d=768, level_bits=(10, 13, 16, 19), branchings=(0, 32, 32, 32), active=(8, 8, 8, 32)),
    "b64": dict(d=1024, level_bits=(10, 13, 16, 20), branchings=(0, 64, 64, 64), active=(4, 4, 8, 32)),
}


def _branchy(hname):
    h = NARROW_BRANCHY[hname]
    d, nb, dl, K = h["d"], list(h["level_bits"]), list(h["branchings"]), list(h["active"])
    plan = dpb.Plan(d, seed=0, level_bits=nb, branchings=dl, active=K)
    assert dpb.load().dpb_encode_workspace_bytes(plan._handle, 100) == 0   # the narrow encoder runs it
    return plan, d, nb, dl, K, oracle.masks(d, nb[-1]), oracle.generators(nb, dl, 0)


@pytest.mark.parametrize("hname,T", [("k2", 64), ("k2", 33), ("b32", 200), ("b32", 31), ("b64", 150)])
def test_encode_narrow_many_children_per_parent(hname, T):
    say(f"[encode branchy] {hname} T={T}")
    plan, d, nb, dl, K, m, gens = _branchy(hname)
    x = inputs.normal((T, d), 1100 + T + len(hname), "bf16")
    idx, coef = dpb.encode(plan, x.to(DEV))
    torch.cuda.synchronize()
    oi, oc, om, oo = oracle.encode(d, m, nb, K, dl, gens, x.double().numpy())
    st = compare_encode(K, idx.cpu().numpy(), coef.cpu().numpy(), oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(d, m, gens, x.double().numpy()))
    say(f"  {st}")
    assert st["exempt_tokens"] <= max(2, 0.02 * T)
    assert (idx.cpu().numpy() >= 0).all()   # every level has enough candidates: no padding


def test_encode_one_lane_holds_eight_keys_above_threshold():
    """A token whose level-1 top 8 are exactly the 8 children one lane of the
    matrix-core layout holds (generators 0-3 and 16-19 of one parent column),
    so that lane counts 8 keys at or above the threshold."""
    say("[encode branchy crafted] b32")
    plan, d, nb, dl, K, m, gens = _branchy("b32")
    x = inputs.normal((6, d), 1200, "bf16").double().numpy() * 0.05
    p = 123
    lane_rows = [0, 1, 2, 3, 16, 17, 18, 19]
    kids = [p ^ int(gens[1][j]) for j in lane_rows]
    for t in (0, 3):
        x[t, p] = 8.0
        for c in kids:
            x[t] += 3.0 * oracle.phi(d, m, c)
    xb = torch.from_numpy(x).to(torch.bfloat16)
    idx, coef = dpb.encode(plan, xb.to(DEV))
    torch.cuda.synchronize()
    oi, oc, om, oo = oracle.encode(d, m, nb, K, dl, gens, xb.double().numpy())
    for t in (0, 3):
        assert oi[t, 0] == p and sorted(oi[t, K[0]:K[0] + K[1]].tolist()) == sorted(kids)
    st = compare_encode(K, idx.cpu().numpy(), coef.cpu().numpy(), oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(d, m, gens, xb.double().numpy()))
    say(f"  {st}")
    assert sorted(idx.cpu().numpy()[0, K[0]:K[0] + K[1]].tolist()) == sorted(kids)


def test_encode_dyadic_ties_tiny():
    """Integer activations: hashed scores are multiples of 1/8 and tie often;
    fp32 sums are exact, so selection must match exactly with index tie-breaks."""
    say("[encode dyadic] tiny")
    plan = plan_for("tiny")
    w, nb, dl, K, m, gens = oracle_setup("tiny")
    x = inputs.dyadic(w.d, 256)
    idx, coef = dpb.encode(plan, x.to(DEV))
    torch.cuda.synchronize()
    oi, oc, _, _ = oracle.encode(w.d, m, nb, K, dl, gens, x.double().numpy())
    assert np.array_equal(idx.cpu().numpy(), oi)
    assert np.array_equal(coef.cpu().numpy().astype(np.float64), oc)


def test_encode_deterministic_and_empty():
    say("[encode determinism] gpt2")
    plan = plan_for("gpt2")
    x = inputs.activations("gpt2", 2048).to(DEV)
    a = dpb.encode(plan, x)
    b = dpb.encode(plan, x)
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
    e = dpb.encode(plan, x[:0])
    assert e[0].shape == (0, plan.k_tot)


# ---------------------------------------------------------------- decode

def _oracle_codes(name, T):
    w, nb, dl, K, m, gens = oracle_setup(name)
    x = inputs.activations(name, T)
    oi, oc, _, _ = oracle.encode(w.d, m, nb, K, dl, gens, x.double().numpy())
    return w, m, oi, oc.astype(np.float32)


@pytest.mark.parametrize("name,T", [("tiny", 256), ("gpt2", 777), ("wide", 300), ("wide", 301), ("very_wide", 130)])
@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_decode_matches_oracle(name, T, out):
    say(f"[decode] {name} T={T} out={out}")
    plan = plan_for(name)
    w, m, oi, oc = _oracle_codes(name, T)
    dt = torch.float32 if out == "f32" else torch.bfloat16
    y = dpb.decode(plan, torch.from_numpy(oi).to(DEV), torch.from_numpy(oc).to(DEV), dt)
    torch.cuda.synchronize()
    ref = oracle.decode(w.d, m, oi, oc.astype(np.float64))
    err = compare_dense(y.float().cpu().numpy(), ref, TOL_F32 if out == "f32" else TOL_BF16)
    say(f"  max rel err {err:.3g}")


@pytest.mark.parametrize("name", ["tiny", "wide", "very_wide"])
def test_decode_arbitrary_codes(name):
    """Any valid code, not only encoder output: indices anywhere in the
    dictionary, repeated indices, basis slots and padding."""
    say(f"[decode arbitrary] {name}")
    plan = plan_for(name)
    w = inputs.workload(name)
    m = oracle.masks(w.d, w.n)
    T, k = 97, plan.k_tot
    rng = np.random.default_rng(11)
    idx = rng.integers(0, 1 << w.n, size=(T, k)).astype(np.int32)
    idx[:, :3] = rng.integers(0, w.d, size=(T, 3))
    idx[::4, 1] = idx[::4, 0]          # a basis coordinate held twice
    idx[:, 5] = idx[:, 6]
    idx[::3, -2:] = -1
    coef = rng.standard_normal((T, k)).astype(np.float32)
    y = dpb.decode(plan, torch.from_numpy(idx).to(DEV), torch.from_numpy(coef).to(DEV))
    torch.cuda.synchronize()
    ref = oracle.decode(w.d, m, idx, coef.astype(np.float64))
    compare_dense(y.cpu().numpy(), ref, TOL_F32)


def _mixed_codes(name, T, seed=21):
    """Encoder codes with edits: a repeated last-level slot (two slots compete
    for one parent column), unroutable indices, a basis index in a hashed
    level, a hashed index in level 0, and padding in the last level, among
    its parents and below them."""
    w, m, oi, oc = _oracle_codes(name, T)
    nb, _, K = oracle.hierarchy(w.d, w.n, w.levels, w.branching, w.beam, w.k)
    rng = np.random.default_rng(seed)
    idx, coef = oi.copy(), oc.copy()
    last = sum(K[:-1])
    idx[::2, last + 3] = idx[::2, last + 2]
    idx[1::3, last + 5] = rng.integers(1 << nb[-2], 1 << nb[-1], size=idx[1::3].shape[0])
    idx[::4, last + 1] = -1
    idx[::5, K[0]] = rng.integers(0, w.d, size=idx[::5].shape[0])
    idx[::7, 1] = rng.integers(w.d, 1 << w.n, size=idx[::7].shape[0])
    idx[3::7, 2] = idx[3::7, 0]        # a basis coordinate held twice
    lp = sum(K[:-2])                   # first slot of the last level's parents
    idx[2::6, lp + 1] = -1             # padding among the last level's parents
    if len(K) >= 4:
        idx[5::8, K[0] + 1] = -1       # padding in a level below them
    coef[:, last + 4] *= -3.0
    return w, m, idx, coef


@pytest.mark.parametrize("name", ["tiny", "gpt2", "wide", "very_wide"])
def test_decode_and_bwd_mixed_codes(name):
    say(f"[decode+bwd mixed] {name}")
    plan = plan_for(name)
    w, m, idx, coef = _mixed_codes(name, 90)
    di = torch.from_numpy(idx).to(DEV)
    y = dpb.decode(plan, di, torch.from_numpy(coef).to(DEV))
    g = inputs.upstream_grad(name, 90)
    gc, gx = dpb.decode_bwd(plan, di, g.to(DEV), torch.float32)
    torch.cuda.synchronize()
    compare_dense(y.cpu().numpy(), oracle.decode(w.d, m, idx, coef.astype(np.float64)), TOL_F32)
    rgc, rgx = oracle.decode_bwd(w.d, m, idx, g.double().numpy())
    compare_dense(gc.cpu().numpy(), rgc, TOL_F32)
    compare_dense(gx.cpu().numpy(), rgx, TOL_F32)


@pytest.mark.parametrize("name", ["wide", "very_wide"])
def test_decode_and_bwd_deterministic(name):
    """Two launches on the same codes (with repeated coordinates and slots)
    give the same bits: lanes that write the same LDS word write the same
    value, and repeated coordinates are added in slot order."""
    say(f"[decode+bwd deterministic] {name}")
    plan = plan_for(name)
    w, m, idx, coef = _mixed_codes(name, 301, seed=23)
    di, dc = torch.from_numpy(idx).to(DEV), torch.from_numpy(coef).to(DEV)
    g = inputs.upstream_grad(name, 301).to(DEV)
    y1 = dpb.decode(plan, di, dc)
    y2 = dpb.decode(plan, di, dc)
    gc1, gx1 = dpb.decode_bwd(plan, di, g, torch.float32)
    gc2, gx2 = dpb.decode_bwd(plan, di, g, torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    assert torch.equal(gc1, gc2) and torch.equal(gx1, gx2)
    compare_dense(y1.cpu().numpy(), oracle.decode(w.d, m, idx, coef.astype(np.float64)), TOL_F32)


def test_decode_dyadic_bit_exact_and_one_hot():
    say("[decode exact] tiny")
    plan = plan_for("tiny")
    w = inputs.workload("tiny")
    m = oracle.masks(w.d, w.n)
    rng = np.random.default_rng(3)
    T, k = 64, plan.k_tot
    idx = rng.integers(0, 1 << w.n, size=(T, k)).astype(np.int32)
    coef = rng.integers(-8, 9, size=(T, k)).astype(np.float32)
    y = dpb.decode(plan, torch.from_numpy(idx).to(DEV), torch.from_numpy(coef).to(DEV))
    torch.cuda.synchronize()
    ref = oracle.decode(w.d, m, idx, coef.astype(np.float64))
    assert np.array_equal(y.cpu().numpy().astype(np.float64), ref)
    # one-hot codes of hashed features return exactly +-fp32(1/sqrt d)
    for name in ("tiny", "wide"):
        p = plan_for(name)
        ww = inputs.workload(name)
        oh = np.full((4, p.k_tot), -1, np.int32)
        oh[:, 0] = [ww.d, ww.d + 1, (1 << ww.n) - 1, 12345 % (1 << ww.n) + ww.d]
        c = np.zeros((4, p.k_tot), np.float32)
        c[:, 0] = 1
        yy = dpb.decode(p, torch.from_numpy(oh).to(DEV), torch.from_numpy(c).to(DEV)).cpu().numpy()
        v = np.float32(1.0 / math.sqrt(ww.d))
        assert set(np.unique(yy).tolist()) == {float(v), float(-v)}


@pytest.mark.parametrize("name", ["gpt2", "wide", "very_wide"])
def test_decode_full_size_sampled(name):
    w = inputs.workload(name)
    say(f"[decode full] {name} T={w.tokens}")
    plan = plan_for(name)
    x = full_activations(name).to(DEV)
    idx, coef = dpb.encode(plan, x)
    y = dpb.decode(plan, idx, coef, torch.bfloat16)
    torch.cuda.synchronize()
    r = sample_rows(w.tokens, 256, seed=w.index + 1)
    m = oracle.masks(w.d, w.n)
    ih, ch = idx.cpu().numpy()[r], coef.cpu().numpy()[r].astype(np.float64)
    compare_dense(y.float().cpu().numpy()[r], oracle.decode(w.d, m, ih, ch), TOL_BF16)


# ---------------------------------------------------------------- backward

@pytest.mark.parametrize("name,T", [("tiny", 256), ("gpt2", 500), ("train", 300), ("train", 301), ("very_wide", 120)])
def test_decode_bwd_matches_oracle(name, T):
    say(f"[bwd] {name} T={T}")
    plan = plan_for(name)
    w, m, oi, _ = _oracle_codes(name, T)
    g = inputs.upstream_grad(name, T)
    gc, gx = dpb.decode_bwd(plan, torch.from_numpy(oi).to(DEV), g.to(DEV))
    torch.cuda.synchronize()
    rgc, rgx = oracle.decode_bwd(w.d, m, oi, g.double().numpy())
    tol = TOL_F32 if w.dtype == "f32" else TOL_BF16
    e1 = compare_dense(gc.cpu().numpy(), rgc, TOL_F32)
    e2 = compare_dense(gx.float().cpu().numpy(), rgx, tol)
    say(f"  grad_coef err {e1:.3g}  grad_x err {e2:.3g}")


def test_decode_bwd_full_size_sampled_train():
    w = inputs.workload("train")
    say(f"[bwd full] train T={w.tokens}")
    plan = plan_for("train")
    x = full_activations("train").to(DEV)
    g = inputs.upstream_grad("train").to(DEV)
    idx, coef = dpb.encode(plan, x)
    gc, gx = dpb.decode_bwd(plan, idx, g)
    torch.cuda.synchronize()
    r = sample_rows(w.tokens, 256, seed=9)
    m = oracle.masks(w.d, w.n)
    rgc, rgx = oracle.decode_bwd(w.d, m, idx.cpu().numpy()[r], g.cpu()[r].double().numpy())
    compare_dense(gc.cpu().numpy()[r], rgc, TOL_F32)
    compare_dense(gx.float().cpu().numpy()[r], rgx, TOL_BF16)


def test_decode_bwd_adjoint_identity():
    """<decode(idx, a), g> == <a, grad_coef(idx, g)> (fp32 sums, fp64 compare)."""
    say("[bwd adjoint] wide")
    plan = plan_for("wide")
    w = inputs.workload("wide")
    rng = np.random.default_rng(5)
    T = 64
    idx = torch.from_numpy(rng.integers(0, 1 << w.n, size=(T, plan.k_tot)).astype(np.int32)).to(DEV)
    a = torch.from_numpy(rng.standard_normal((T, plan.k_tot)).astype(np.float32)).to(DEV)
    g = torch.from_numpy(rng.standard_normal((T, w.d)).astype(np.float32)).to(DEV)
    y = dpb.decode(plan, idx, a)
    gc, gx = dpb.decode_bwd(plan, idx, g, torch.float32)
    lhs = (y.double() * g.double()).sum(1)
    rhs = (a.double() * gc.double()).sum(1)
    assert torch.allclose(lhs, rhs, rtol=1e-4, atol=1e-4)
    assert torch.allclose(gx, dpb.decode(plan, idx, gc), rtol=0, atol=0)


def test_boundary_errors_on_gpu():
    say("[errors] gpu")
    plan = plan_for("tiny")
    x = torch.zeros((8, 64), device=DEV)
    with pytest.raises(TypeError):
        dpb.encode(plan, x.half())
    xb = torch.zeros(8 * 64 + 1, device=DEV)[1:].view(8, 64)   # 4-byte offset: misaligned
    with pytest.raises(dpb.DPBError):
        dpb.encode(plan, xb)
