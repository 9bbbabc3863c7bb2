"""GPU parity at dimensions d that are not a multiple of the 32-coordinate
chunk (the last chunk of every row, sign bitmap and table is ragged), some
of them not a multiple of the 8-element vector loads and stores either.

Each plan runs encode, decode (on the oracle's codes) and decode-backward
against the oracle on a ragged number of tokens.  The dictionary for d not a
power of two follows the oracle's reading of the mask construction, which the
library's own tables reproduce bit for bit (test_boundary).
"""
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

# d % 32 != 0 everywhere; d % 8 != 0 for d100 and d522.  "d522" has 32
# children per parent (two generator tiles per level), "wide1000" 256 (the
# wide encoder and the backward's direct reductions).
RAGGED = {
    "d200_f32": dict(d=200, cfg=(12, 3, 16, 4, 8), dtype="f32"),
    "d100": dict(d=100, cfg=(11, 3, 16, 4, 8), dtype="bf16"),
    "d1000": dict(d=1000, cfg=(16, 4, 16, 8, 32), dtype="bf16"),
    "d522": dict(d=522, hier=((10, 13, 16), (0, 32, 32), (8, 8, 16)), dtype="bf16"),
    "wide1000": dict(d=1000, hier=((10, 15), (0, 256), (16, 32)), dtype="bf16"),
}


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    dpb.load()


_SETUP = {}


def setup(name):
    """(plan, d, level bits, branchings, active, masks, generators, dtype)."""
    if name not in _SETUP:
        h = RAGGED[name]
        d = h["d"]
        if "cfg" in h:
            n, L, b, beam, k = h["cfg"]
            nb, dl, K = oracle.hierarchy(d, n, L, b, beam, k)
            plan = dpb.Plan(d, n, L, b, beam, k, 0)
        else:
            nb, dl, K = (list(v) for v in h["hier"])
            plan = dpb.Plan(d, seed=0, level_bits=nb, branchings=dl, active=K)
        _SETUP[name] = (plan, d, nb, dl, K, oracle.masks(d, nb[-1]), oracle.generators(nb, dl, 0), h["dtype"])
    return _SETUP[name]


@pytest.mark.parametrize("name", list(RAGGED))
def test_ragged_dim_encode(name):
    plan, d, nb, dl, K, m, gens, dt = setup(name)
    T = 77
    say(f"[ragged encode] {name} d={d} T={T}")
    # the wide encoder needs a workspace, the narrow one none
    wide = dpb.load().dpb_encode_workspace_bytes(plan._handle, T) > 0
    assert wide == name.startswith("wide")
    x = inputs.normal((T, d), 5100 + d, dt)
    idx, coef = dpb.encode(plan, x.to(DEV))
    torch.cuda.synchronize()
    xd = x.double().numpy()
    oi, oc, om, oo = oracle.encode(d, m, nb, K, dl, gens, xd)
    st = compare_encode(K, idx.cpu().numpy(), coef.cpu().numpy(), oi, oc, om, oo, TOL_F32,
                        ctx=EncodeCheck(d, m, gens, xd))
    say(f"  {st}")
    assert st["exempt_tokens"] <= max(2, 0.02 * T)


@pytest.mark.parametrize("name", list(RAGGED))
def test_ragged_dim_decode_and_bwd(name):
    plan, d, nb, dl, K, m, gens, dt = setup(name)
    T = 45
    say(f"[ragged decode/bwd] {name} d={d} T={T}")
    x = inputs.normal((T, d), 5200 + d, dt)
    oi, oc, _, _ = oracle.encode(d, m, nb, K, dl, gens, x.double().numpy())
    oc32 = oc.astype(np.float32)
    idx = torch.from_numpy(oi).to(DEV)
    tdt = torch.float32 if dt == "f32" else torch.bfloat16
    tol = TOL_F32 if dt == "f32" else TOL_BF16
    y = dpb.decode(plan, idx, torch.from_numpy(oc32).to(DEV), tdt)
    g = inputs.normal((T, d), 5300 + d, dt)
    gc, gx = dpb.decode_bwd(plan, idx, g.to(DEV))
    torch.cuda.synchronize()
    assert y.shape == (T, d) and gx.shape == (T, d)
    ey = compare_dense(y.float().cpu().numpy(), oracle.decode(d, m, oi, oc32.astype(np.float64)), tol)
    rgc, rgx = oracle.decode_bwd(d, m, oi, g.double().numpy())
    e1 = compare_dense(gc.cpu().numpy(), rgc, TOL_F32)
    e2 = compare_dense(gx.float().cpu().numpy(), rgx, tol)
    say(f"  y err {ey:.3g}  grad_coef err {e1:.3g}  grad_x err {e2:.3g}")
