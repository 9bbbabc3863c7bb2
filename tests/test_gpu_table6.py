"""GPU parity on the paper's own hierarchies (App. G, Table 6): d = 1024 or
2048, level bits (10|11, 15[, 17]), K = (16, 32[, 64]), 256 children scored per
active parent.  Same rules as the other parity tests: encode against the
oracle with near-tie exemptions above level 0, decode and backward on the
oracle's codes; full-size runs on sampled rows.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2607_20652_amd import binding as dpb
from paper_2607_20652_amd import inputs
from paper_2607_20652_amd import autograd as dpb_autograd
from parity_util import TOL_BF16, TOL_F32, compare_dense, compare_encode, random_std_state, EncodeCheck

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
NAMES = ["pt_small_2l", "pt_large_2l", "pt_small_3l"]
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
        _PLANS[name] = dpb.Plan(w.d, seed=0, **w.plan_kwargs())
    return _PLANS[name]


def setup(name):
    w = inputs.workload(name)
    nb, dl, K = w.hierarchy()
    return w, nb, dl, K, oracle.masks(w.d, nb[-1]), oracle.generators(nb, dl, 0)


def test_plans_have_table6_shapes():
    for name in NAMES:
        w, nb, dl, K, _, _ = setup(name)
        p = plan_for(name)
        assert (p.level_bits, p.branching, p.active) == (nb, dl, K)
        assert p.k_tot == sum(K)


@pytest.mark.parametrize("name,T", [("pt_small_2l", 96), ("pt_large_2l", 37), ("pt_small_3l", 70)])
def test_encode_matches_oracle(name, T):
    say(f"[t6 encode] {name} T={T}")
    plan = plan_for(name)
    w, nb, dl, K, m, gens = setup(name)
    x = inputs.activations(name, T)
    idx, coef = dpb.encode(plan, x.to(DEV))
    torch.cuda.synchronize()
    oi, oc, om, oo = oracle.encode(w.d, m, nb, K, dl, gens, x.double().numpy())
    st = compare_encode(K, idx.cpu().numpy(), coef.cpu().numpy(), oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(w.d, m, gens, x.double().numpy()))
    say(f"  {st}")
    assert st["exempt_tokens"] <= max(2, 0.02 * T)


@pytest.mark.parametrize("name", NAMES)
def test_encode_full_size_sampled(name):
    w, nb, dl, K, m, gens = setup(name)
    say(f"[t6 encode full] {name} T={w.tokens}")
    plan = plan_for(name)
    x = inputs.activations(name)
    idx, coef = dpb.encode(plan, x.to(DEV))
    torch.cuda.synchronize()
    rng = np.random.default_rng(w.index)
    rows = np.unique(np.concatenate([np.arange(16), rng.choice(w.tokens, 32, replace=False),
                                     np.arange(w.tokens - 16, w.tokens)]))
    oi, oc, om, oo = oracle.encode(w.d, m, nb, K, dl, gens, x[rows].double().numpy())
    st = compare_encode(K, idx.cpu().numpy()[rows], coef.cpu().numpy()[rows], oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(w.d, m, gens, x[rows].double().numpy()))
    say(f"  {st}")
    assert st["exempt_tokens"] <= max(2, 0.02 * len(rows))
    # every emitted index is unique within its token and lies in its level
    ii = idx.cpu().numpy()
    lo = [0] + [1 << b for b in nb[:-1]]
    hi = [w.d] + [1 << b for b in nb[1:]]
    s = 0
    for l, k in enumerate(K):
        blk = ii[:, s:s + k]
        assert ((blk >= lo[l]) & (blk < hi[l])).all()
        srt = np.sort(blk, axis=1)
        assert (srt[:, 1:] != srt[:, :-1]).all()
        s += k


@pytest.mark.parametrize("name,T", [("pt_small_2l", 130), ("pt_large_2l", 50), ("pt_small_3l", 90)])
@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_decode_and_bwd_match_oracle(name, T, out):
    say(f"[t6 decode+bwd] {name} T={T} {out}")
    plan = plan_for(name)
    w, nb, dl, K, m, gens = setup(name)
    x = inputs.activations(name, T)
    oi, oc, _, _ = oracle.encode(w.d, m, nb, K, dl, gens, x.double().numpy())
    dt = torch.float32 if out == "f32" else torch.bfloat16
    tol = TOL_F32 if out == "f32" else TOL_BF16
    di = torch.from_numpy(oi).to(DEV)
    y = dpb.decode(plan, di, torch.from_numpy(oc.astype(np.float32)).to(DEV), dt)
    g = inputs.upstream_grad(name, T)
    gc, gx = dpb.decode_bwd(plan, di, g.to(DEV), dt)
    torch.cuda.synchronize()
    compare_dense(y.float().cpu().numpy(), oracle.decode(w.d, m, oi, oc.astype(np.float32).astype(np.float64)), tol)
    rgc, rgx = oracle.decode_bwd(w.d, m, oi, g.double().numpy())
    compare_dense(gc.cpu().numpy(), rgc, TOL_F32)
    compare_dense(gx.float().cpu().numpy(), rgx, tol)


@pytest.mark.parametrize("name,T", [("pt_small_2l", 60), ("pt_small_3l", 40)])
def test_encode_std_matches_oracle(name, T):
    """The wide encoder on standardized scores (random EMA statistics)."""
    say(f"[t6 encode std] {name} T={T}")
    plan = plan_for(name)
    w, nb, dl, K, m, gens = setup(name)
    N = 1 << nb[-1]
    mu, _, r = random_std_state(N, 77 + w.index)
    stats = torch.from_numpy(np.stack([mu, r], axis=1)).contiguous().to(DEV)
    x = inputs.activations(name, T)
    idx, coef = dpb.encode_std(plan, x.to(DEV), stats)
    torch.cuda.synchronize()
    oi, oc, om, oo = oracle.encode_std(w.d, m, nb, K, dl, gens, x.double().numpy(), mu, r)
    st = compare_encode(K, idx.cpu().numpy(), coef.cpu().numpy(), oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(w.d, m, gens, x.double().numpy(), mu, r))
    say(f"  {st}")
    assert st["exempt_tokens"] <= max(2, 0.02 * T)


@pytest.mark.parametrize("name,T,beta", [("pt_small_2l", 300, 0.1), ("pt_small_3l", 160, 0.05)])
def test_std_update_matches_oracle(name, T, beta):
    """The EMA update of the statistics at the paper's own shapes (K_{l-1}
    Delta_l = 4096 and 8192 candidates per sampled token)."""
    say(f"[t6 std update] {name} T={T} beta={beta}")
    plan = plan_for(name)
    w, nb, dl, K, m, gens = setup(name)
    N = 1 << nb[-1]
    mu, m2, r = random_std_state(N, 61 + w.index)
    stats = torch.from_numpy(np.stack([mu, r], axis=1)).contiguous().to(DEV)
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
    assert touched[w.d:].sum() > 4 * K[0] * dl[1]   # level >= 1 features of the sampled tokens
    assert np.array_equal(gs[~touched], before.cpu().numpy()[~touched])
    assert np.array_equal(gv[~touched], m2[~touched])
    assert np.allclose(gs[touched, 0], rmu[touched], rtol=1e-5, atol=1e-5)
    assert np.allclose(gv[touched], rm2[touched], rtol=1e-5, atol=1e-5)
    rr = oracle.std_r(gs[touched, 0].astype(np.float64), gv[touched].astype(np.float64), 1e-6)
    assert np.allclose(gs[touched, 1], rr, rtol=2e-6, atol=0)


@pytest.mark.parametrize("name,T", [("pt_small_2l", 128), ("pt_small_3l", 96)])
def test_standardized_layer_step(name, T):
    """One training step of the DPB layer on standardized scores at the
    paper's own shapes: forward and input gradient against the oracle, and
    the statistics update the backward applies."""
    say(f"[t6 std layer] {name} T={T}")
    plan = plan_for(name)
    w, nb, dl, K, m, gens = setup(name)
    N = 1 << nb[-1]
    std = dpb_autograd.Standardizer(plan, momentum=0.1, eps=1e-6)
    mu, m2, r = random_std_state(N, 71 + w.index)
    std.stats.copy_(torch.from_numpy(np.stack([mu, r], axis=1)))
    std.m2.copy_(torch.from_numpy(m2))
    x = inputs.activations(name, T).to(DEV).requires_grad_(True)
    gy = inputs.upstream_grad(name, T).to(DEV)
    y, lv = dpb_autograd.dpb_layer(x, plan, True, 2, std)
    stats0 = torch.from_numpy(np.stack([mu, r], axis=1)).contiguous().to(DEV)
    idx, coef = dpb.encode_std(plan, x.detach(), stats0)
    torch.autograd.backward([y, lv], [gy, torch.tensor(0.5, device=DEV)])
    torch.cuda.synchronize()
    ii, cc = idx.cpu().numpy(), coef.cpu().numpy().astype(np.float64)
    oi, oc, om, oo = oracle.encode_std(w.d, m, nb, K, dl, gens, x.detach().double().cpu().numpy(), mu, r)
    st = compare_encode(K, ii, cc, oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(w.d, m, gens, x.detach().double().cpu().numpy(), mu, r))
    say(f"  {st}")
    xd = x.detach().double().cpu().numpy()
    ry, _ = oracle.normalize(oracle.decode(w.d, m, ii, cc), xd)
    compare_dense(y.detach().float().cpu().numpy(), ry, TOL_BF16)
    rs = np.where(ii >= 0, r[np.maximum(ii, 0)], 0.0)
    _, rgx = oracle.layer_backward(w.d, m, ii, cc, xd, gy.double().cpu().numpy(), 0.5, 2, True, r_slot=rs)
    compare_dense(x.grad.float().cpu().numpy(), rgx, TOL_BF16)
    rmu, rm2 = oracle.std_update(w.d, m, nb, K, dl, gens, xd, ii, mu.astype(np.float64), m2.astype(np.float64), 0.1)
    assert np.allclose(std.stats.cpu().numpy()[:, 0], rmu, rtol=1e-5, atol=1e-5)
    assert np.allclose(std.m2.cpu().numpy(), rm2, rtol=1e-5, atol=1e-5)


def test_encode_zero_and_constant_rows():
    """Degenerate rows: all-zero activations (every score 0, ties broken by
    index) and a constant row, through the wide encoder's threshold and
    fallback paths."""
    name = "pt_small_2l"
    say(f"[t6 encode degenerate] {name}")
    plan = plan_for(name)
    w, nb, dl, K, m, gens = setup(name)
    x = inputs.activations(name, 8).clone()
    x[0] = 0
    x[3] = 0.5
    x[5, : w.d // 2] = 0
    idx, coef = dpb.encode(plan, x.to(DEV))
    torch.cuda.synchronize()
    oi, oc, om, oo = oracle.encode(w.d, m, nb, K, dl, gens, x.double().numpy())
    st = compare_encode(K, idx.cpu().numpy(), coef.cpu().numpy(), oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(w.d, m, gens, x.double().numpy()))
    say(f"  {st}")
    assert np.array_equal(idx.cpu().numpy()[0], oi[0])
    assert st["exempt_tokens"] <= 2


@pytest.mark.parametrize("name,T", [("pt_small_2l", 50), ("pt_small_3l", 33)])
def test_encode_f32_input_matches_oracle(name, T):
    """fp32 activations: the wide GEMM splits each value into three bf16 terms."""
    say(f"[t6 encode f32] {name} T={T}")
    plan = plan_for(name)
    w, nb, dl, K, m, gens = setup(name)
    x = inputs.normal((T, w.d), 500 + w.index)
    idx, coef = dpb.encode(plan, x.to(DEV))
    torch.cuda.synchronize()
    oi, oc, om, oo = oracle.encode(w.d, m, nb, K, dl, gens, x.double().numpy())
    st = compare_encode(K, idx.cpu().numpy(), coef.cpu().numpy(), oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(w.d, m, gens, x.double().numpy()))
    say(f"  {st}")
    assert st["exempt_tokens"] <= max(2, 0.02 * T)


@pytest.mark.parametrize("name,T", [("pt_small_2l", 45), ("pt_small_3l", 29)])
def test_decode_bwd_f32_grad_matches_oracle(name, T):
    """fp32 upstream gradient through the direct reductions of wide plans."""
    say(f"[t6 bwd f32 g] {name} T={T}")
    plan = plan_for(name)
    w, nb, dl, K, m, gens = setup(name)
    x = inputs.activations(name, T)
    oi, _, _, _ = oracle.encode(w.d, m, nb, K, dl, gens, x.double().numpy())
    g = inputs.normal((T, w.d), 600 + w.index)
    gc, gx = dpb.decode_bwd(plan, torch.from_numpy(oi).to(DEV), g.to(DEV), torch.float32)
    torch.cuda.synchronize()
    rgc, rgx = oracle.decode_bwd(w.d, m, oi, g.double().numpy())
    compare_dense(gc.cpu().numpy(), rgc, TOL_F32)
    compare_dense(gx.cpu().numpy(), rgx, TOL_F32)


CHUNK = 16384   # tokens per pass of the wide encoder


def test_encode_chunk_boundary_and_full_chunks():
    """More than one chunk of the wide encoder with a ragged last chunk:
    sampled rows on both sides of each chunk boundary."""
    name = "pt_small_2l"
    T = 2 * CHUNK + 77
    say(f"[t6 encode chunks] {name} T={T}")
    plan = plan_for(name)
    w, nb, dl, K, m, gens = setup(name)
    x = inputs.normal((T, w.d), 900, "bf16")
    idx, coef = dpb.encode(plan, x.to(DEV))
    torch.cuda.synchronize()
    rows = np.array([0, 1, CHUNK - 2, CHUNK - 1, CHUNK, CHUNK + 1, 2 * CHUNK - 2, 2 * CHUNK - 1, 2 * CHUNK,
                     2 * CHUNK + 1, T - 2, T - 1])
    oi, oc, om, oo = oracle.encode(w.d, m, nb, K, dl, gens, x[rows].double().numpy())
    st = compare_encode(K, idx.cpu().numpy()[rows], coef.cpu().numpy()[rows], oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(w.d, m, gens, x[rows].double().numpy()))
    say(f"  {st}")
    assert st["exempt_tokens"] <= 2


# Wide hierarchies beyond Table 6, for the encoder's other tile shapes: 128 and
# 64 children per parent (4 and 2 row tiles per wave), 48 parents per token
# (one token per 64-column wave tile), and a level of 16 children inside a
# wide plan (padding generator rows, scores written in full).
CUSTOM = {
    "wide_mixed": dict(d=1024, level_bits=(10, 14, 17), branchings=(0, 128, 64), active=(16, 48, 40)),
    "wide_small_delta": dict(d=1024, level_bits=(10, 15, 19), branchings=(0, 256, 16), active=(16, 32, 64)),
}


@pytest.mark.parametrize("hname,T", [("wide_mixed", 70), ("wide_small_delta", 50)])
def test_custom_wide_hierarchies(hname, T):
    h = CUSTOM[hname]
    d, nb, dl, K = h["d"], list(h["level_bits"]), list(h["branchings"]), list(h["active"])
    say(f"[wide custom] {hname} T={T}")
    plan = dpb.Plan(d, seed=0, level_bits=nb, branchings=dl, active=K)
    m, gens = oracle.masks(d, nb[-1]), oracle.generators(nb, dl, 0)
    x = inputs.normal((T, d), 700 + len(hname), "bf16")
    idx, coef = dpb.encode(plan, x.to(DEV))
    torch.cuda.synchronize()
    oi, oc, om, oo = oracle.encode(d, m, nb, K, dl, gens, x.double().numpy())
    st = compare_encode(K, idx.cpu().numpy(), coef.cpu().numpy(), oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(d, m, gens, x.double().numpy()))
    say(f"  {st}")
    assert st["exempt_tokens"] <= max(2, 0.02 * T)
    g = inputs.normal((T, d), 800 + len(hname), "bf16")
    gc, gx = dpb.decode_bwd(plan, torch.from_numpy(oi).to(DEV), g.to(DEV), torch.float32)
    y = dpb.decode(plan, torch.from_numpy(oi).to(DEV), torch.from_numpy(oc.astype(np.float32)).to(DEV),
                   torch.float32)
    torch.cuda.synchronize()
    rgc, rgx = oracle.decode_bwd(d, m, oi, g.double().numpy())
    compare_dense(gc.cpu().numpy(), rgc, TOL_F32)
    compare_dense(gx.cpu().numpy(), rgx, TOL_F32)
    compare_dense(y.cpu().numpy(), oracle.decode(d, m, oi, oc.astype(np.float32).astype(np.float64)), TOL_F32)


def test_encode_rejects_missing_or_small_workspace():
    """A plan that needs a workspace (many children per parent) and is given
    none, or too little, is refused on the host before anything is enqueued."""
    import ctypes
    name, T = "pt_small_3l", 24
    say(f"[t6 encode small workspace] {name} T={T}")
    plan = plan_for(name)
    x = inputs.activations(name, T).to(DEV)
    assert dpb.load().dpb_encode_workspace_bytes(plan._handle, T) > 0
    idx = torch.full((T, plan.k_tot), 7, dtype=torch.int32, device=DEV)
    coef = torch.zeros((T, plan.k_tot), dtype=torch.float32, device=DEV)
    tiny = torch.empty(4, dtype=torch.float32, device=DEV)
    with pytest.raises(dpb.DPBError) as e:
        dpb.encode(plan, x, idx, coef, workspace=tiny)
    assert e.value.status == -1
    P = ctypes.c_void_p
    st = dpb.load().dpb_encode(plan._handle, P(x.data_ptr()), 1, T, P(idx.data_ptr()), P(coef.data_ptr()), None, 0,
                               None)
    assert st == -1
    torch.cuda.synchronize()
    assert (idx == 7).all().item()


def test_empty_batches():
    name = "pt_small_2l"
    say(f"[t6 empty] {name}")
    plan = plan_for(name)
    w = inputs.workload(name)
    x = torch.empty((0, w.d), dtype=torch.bfloat16, device=DEV)
    idx, coef = dpb.encode(plan, x)
    y = dpb.decode(plan, idx, coef, torch.bfloat16)
    gc, gx = dpb.decode_bwd(plan, idx, torch.empty((0, w.d), dtype=torch.bfloat16, device=DEV), torch.bfloat16)
    torch.cuda.synchronize()
    assert idx.shape == (0, plan.k_tot) and y.shape == (0, w.d) and gc.shape == (0, plan.k_tot)


@pytest.mark.parametrize("name", ["pt_small_3l", "pt_large_2l"])
def test_decode_and_bwd_full_size_sampled(name):
    """The step at its full size (16,384 tokens, the benchmarked launch):
    encode on the GPU, decode and backward of its codes, sampled rows against
    the oracle's decode and backward of the same codes."""
    w, nb, dl, K, m, gens = setup(name)
    say(f"[t6 decode+bwd full] {name} T={w.tokens}")
    plan = plan_for(name)
    x = inputs.activations(name).to(DEV)
    g = inputs.upstream_grad(name).to(DEV)
    idx, coef = dpb.encode(plan, x)
    y = dpb.decode(plan, idx, coef, torch.bfloat16)
    gc, gx = dpb.decode_bwd(plan, idx, g, torch.bfloat16)
    torch.cuda.synchronize()
    rng = np.random.default_rng(5 + w.index)
    rows = np.unique(np.concatenate([np.arange(8), rng.choice(w.tokens, 24, replace=False),
                                     np.arange(w.tokens - 8, w.tokens)]))
    ii, cc = idx.cpu().numpy()[rows], coef.cpu().numpy()[rows].astype(np.float64)
    compare_dense(y.float().cpu().numpy()[rows], oracle.decode(w.d, m, ii, cc), TOL_BF16)
    rgc, rgx = oracle.decode_bwd(w.d, m, ii, g.double().cpu().numpy()[rows])
    compare_dense(gc.cpu().numpy()[rows], rgc, TOL_F32)
    compare_dense(gx.float().cpu().numpy()[rows], rgx, TOL_BF16)


@pytest.mark.parametrize("name", ["pt_small_2l", "pt_small_3l"])
def test_wide_encode_deterministic(name):
    """The GEMM epilogue reserves each wave's list space with an LDS atomic, so
    the order of a token's listed candidates can differ from run to run; the
    selection sorts them, so the code may not.  Plain and standardized scores,
    three runs each, 3,000 tokens (a partial last tile of the level GEMMs)."""
    say(f"[t6 determinism] {name}")
    plan = plan_for(name)
    w = inputs.workload(name)
    x = inputs.activations(name, 3000).to(DEV)
    N = 1 << plan.level_bits[-1]
    mu, _, r = random_std_state(N, 55 + w.index)
    stats = torch.from_numpy(np.stack([mu, r], axis=1)).contiguous().to(DEV)
    for st in (None, stats):
        runs = [dpb.encode(plan, x, stats=st) for _ in range(3)]
        torch.cuda.synchronize()
        for idx, coef in runs[1:]:
            assert torch.equal(idx, runs[0][0])
            assert torch.equal(coef.view(torch.int32), runs[0][1].view(torch.int32))
