"""The allocation-free encoder entry point (dpb_encode_noalloc) through the C
ABI: two calls in a row, the second on a smaller batch, each bit-identical
to dpb_encode / dpb_encode_std with a caller workspace.  The wide plans go
through the library's per-device scratch in several passes; no device memory
is allocated by the calls."""
import sys

import numpy as np
import pytest
import torch

from paper_2607_20652_amd import binding as dpb
from paper_2607_20652_amd import inputs
from parity_util import random_std_state

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


def _plan(name):
    w = inputs.workload(name)
    if name.startswith("pt_"):
        return w, dpb.Plan(w.d, seed=0, **w.plan_kwargs())
    return w, dpb.Plan(w.d, w.n, w.levels, w.branching, w.beam, w.k, 0)


@pytest.mark.parametrize("name,sizes,std", [("pt_small_3l", (4000, 1000), False),
                                            ("pt_small_2l", (2500, 300), True),
                                            ("train", (3000, 257), False)])
def test_noalloc_encode_equals_encode(name, sizes, std):
    w, plan = _plan(name)
    stats = None
    if std:
        mu, _, r = random_std_state(1 << plan.level_bits[-1], 5)
        stats = torch.from_numpy(np.stack([mu, r], axis=1)).contiguous().to(DEV)
    for i, T in enumerate(sizes):
        say(f"[noalloc] {name} call {i} T={T} std={std}")
        x = inputs.normal((T, w.d), 1300 + i, "bf16").to(DEV)
        ref_i, ref_c = dpb.encode(plan, x, stats=stats)
        idx = torch.full((T, plan.k_tot), -7, dtype=torch.int32, device=DEV)
        coef = torch.full((T, plan.k_tot), 7.0, dtype=torch.float32, device=DEV)
        torch.cuda.synchronize()
        free0, _ = torch.cuda.mem_get_info()
        dpb.encode_noalloc(plan, x, idx, coef, stats)
        torch.cuda.synchronize()
        free1, _ = torch.cuda.mem_get_info()
        assert free1 == free0
        assert torch.equal(idx, ref_i)
        assert torch.equal(coef, ref_c)
