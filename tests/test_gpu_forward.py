"""GPU: the forward call (dpb_forward) against the two calls it stands for and
against the oracle.

dpb_forward is specified as dpb_encode (or dpb_encode_std) followed by
dpb_decode of the code just written, so its code and its y must equal those
calls' outputs bit for bit.  The oracle then checks its outputs directly: the
code with the encoder's parity rule, y as the decode of that code.
"""
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


def two_calls(plan, x, stats=None, out_dtype=None):
    idx, coef = dpb.encode(plan, x, stats=stats)
    y = dpb.decode(plan, idx, coef, out_dtype or x.dtype)
    return idx, coef, y


def same(a, b):
    return torch.equal(a.view(torch.int32) if a.dtype == torch.float32 else a.view(torch.int16),
                       b.view(torch.int32) if b.dtype == torch.float32 else b.view(torch.int16))


# ragged token counts: partial groups of two tokens, a group count that is not
# a multiple of the workgroup's waves, and one token
@pytest.mark.parametrize("name,T", [("tiny", 256), ("tiny", 1), ("gpt2", 777), ("wide", 301), ("train", 300),
                                    ("very_wide", 131), ("pt_small_2l", 50)])
def test_forward_equals_encode_then_decode(name, T):
    say(f"[forward] {name} T={T}")
    plan = plan_for(name)
    x = inputs.activations(name, T).to(DEV)
    idx, coef, y = dpb.forward(plan, x)
    ri, rc, ry = two_calls(plan, x)
    torch.cuda.synchronize()
    assert torch.equal(idx, ri)
    assert same(coef, rc)
    assert same(y, ry)


@pytest.mark.parametrize("name,T", [("gpt2", 300), ("train", 257), ("very_wide", 77), ("tiny", 100)])
def test_forward_std_equals_encode_std_then_decode(name, T):
    say(f"[forward std] {name} T={T}")
    plan = plan_for(name)
    w = inputs.workload(name)
    N = 1 << plan.level_bits[-1]
    mu, _, r = random_std_state(N, 91 + w.index)
    stats = torch.from_numpy(np.stack([mu, r], axis=1)).contiguous().to(DEV)
    x = inputs.activations(name, T).to(DEV)
    idx, coef, y = dpb.forward(plan, x, stats=stats)
    ri, rc, ry = two_calls(plan, x, stats=stats)
    torch.cuda.synchronize()
    assert torch.equal(idx, ri)
    assert same(coef, rc)
    assert same(y, ry)


def test_forward_fp32_output_of_bf16_input():
    """y may have another element type than x."""
    plan = plan_for("gpt2")
    x = inputs.activations("gpt2", 130).to(DEV)
    idx, coef, y = dpb.forward(plan, x, out_dtype=torch.float32)
    ri, rc, ry = two_calls(plan, x, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert y.dtype == torch.float32
    assert torch.equal(idx, ri) and same(coef, rc) and same(y, ry)


@pytest.mark.parametrize("name,T", [("gpt2", 200), ("train", 160), ("tiny", 256)])
def test_forward_matches_oracle(name, T):
    say(f"[forward oracle] {name} T={T}")
    plan = plan_for(name)
    w = inputs.workload(name)
    nb, dl, K = oracle.hierarchy(w.d, w.n, w.levels, w.branching, w.beam, w.k)
    m = oracle.masks(w.d, w.n)
    gens = oracle.generators(nb, dl, 0)
    xc = inputs.activations(name, T)
    idx, coef, y = dpb.forward(plan, xc.to(DEV))
    torch.cuda.synchronize()
    xd = xc.double().numpy()
    oi, oc, om, oo = oracle.encode(w.d, m, nb, K, dl, gens, xd)
    tol = TOL_BF16 if w.dtype == "bf16" else TOL_F32
    st = compare_encode(K, idx.cpu().numpy(), coef.cpu().numpy(), oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(w.d, m, gens, xd))
    say(f"  {st}")
    # y is the decode of the GPU's own code
    ry = oracle.decode(w.d, m, idx.cpu().numpy(), coef.cpu().numpy().astype(np.float64))
    compare_dense(y.float().cpu().numpy(), ry, tol)


def test_forward_full_size_train_sampled():
    """The train workload at full size (65,536 tokens): the outputs equal the
    two calls everywhere, and the oracle checks a sample of rows of y against
    the decode of the GPU's code."""
    name = "train"
    plan = plan_for(name)
    w = inputs.workload(name)
    x = inputs.activations(name).to(DEV)
    idx, coef, y = dpb.forward(plan, x)
    ri, rc, ry = two_calls(plan, x)
    torch.cuda.synchronize()
    assert torch.equal(idx, ri) and same(coef, rc) and same(y, ry)
    rows = np.random.Generator(np.random.PCG64(11)).choice(w.tokens, 96, replace=False)
    m = oracle.masks(w.d, w.n)
    ih, ch = idx.cpu().numpy()[rows], coef.cpu().numpy()[rows]
    compare_dense(y.float().cpu().numpy()[rows], oracle.decode(w.d, m, ih, ch.astype(np.float64)), TOL_BF16)


def test_forward_empty_and_errors():
    plan = plan_for("gpt2")
    x = torch.empty((0, plan.d), dtype=torch.bfloat16, device=DEV)
    idx, coef, y = dpb.forward(plan, x)
    assert idx.shape == (0, plan.k_tot) and y.shape == (0, plan.d)
    lib = dpb.load()
    xb = inputs.activations("gpt2", 4).to(DEV)
    i4 = torch.empty((4, plan.k_tot), dtype=torch.int32, device=DEV)
    c4 = torch.empty((4, plan.k_tot), dtype=torch.float32, device=DEV)
    st = lib.dpb_forward(plan._handle, xb.data_ptr(), 1, 4, None, i4.data_ptr(), c4.data_ptr(), None, 1, None, 0,
                         None)
    assert st == -1   # y missing
