"""CPU tests of the C ABI: exports, host tables against the oracle, argument checks.

No compute call runs here (no GPU): error paths that the host detects before
any launch, and the host-only table construction, are what these cover.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2607_20652_amd import binding, inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(binding.lib_path):
        from paper_2607_20652_amd import build
        build.build()
    return binding.load()


def test_exports_every_declared_symbol(lib):
    header = open(os.path.join(ROOT, "include", "dpb.h")).read()
    declared = set(re.findall(r"\b(dpb_[a-z_]+)\s*\(", header))
    assert {"dpb_encode", "dpb_decode", "dpb_decode_bwd", "dpb_plan_create"} <= declared
    for name in declared:
        assert hasattr(lib, name), name


@pytest.mark.parametrize("name", list(inputs.WORKLOADS))
def test_hierarchy_matches_oracle(lib, name):
    w = inputs.workload(name)
    got = binding.hierarchy(w.d, w.n, w.levels, w.branching, w.beam, w.k)
    want = oracle.hierarchy(w.d, w.n, w.levels, w.branching, w.beam, w.k)
    assert got == tuple(want) or list(got) == list(want)


@pytest.mark.parametrize("name", list(inputs.WORKLOADS))
@pytest.mark.parametrize("seed", [0, 12345])
def test_tables_match_oracle_bit_exactly(lib, name, seed):
    w = inputs.workload(name)
    nb, br, _ = oracle.hierarchy(w.d, w.n, w.levels, w.branching, w.beam, w.k)
    m, g = binding.build_tables(w.d, nb, br, seed)
    assert np.array_equal(np.array(m, np.uint32), oracle.masks(w.d, w.n))
    og = oracle.generators(nb, br, seed)
    assert np.array_equal(np.array(g, np.uint32), np.concatenate(og[1:]))


@pytest.mark.parametrize("d,n", [(2, 2), (3, 4), (64, 12), (100, 14), (256, 16), (1000, 20), (2048, 22), (4096, 30)])
def test_masks_match_oracle_other_widths(lib, d, n):
    t = oracle.ceil_log2(d)
    m, _ = binding.build_tables(d, [t, n], [0, 1], 0)
    assert np.array_equal(np.array(m, np.uint32), oracle.masks(d, n))


def _create(lib, *args):
    h = ctypes.c_void_p()
    st = lib.dpb_plan_create(ctypes.byref(h), *args)
    if st == 0:
        lib.dpb_plan_destroy(h)
    return st


@pytest.mark.parametrize("args,status", [
    ((1, 12, 3, 16, 4, 8, 0), -1),        # d < 2
    ((64, 12, 0, 16, 4, 8, 0), -1),       # no levels
    ((64, 12, 9, 16, 4, 8, 0), -1),       # too many levels
    ((64, 31, 3, 16, 4, 8, 0), -1),       # index wider than 30 bits
    ((64, 12, 3, 16, 65, 8, 0), -1),      # K_0 > d
    ((64, 12, 3, 16, 4, 65, 0), -1),      # K_2 > K_1 * Delta_2
    ((64, 12, 3, 0, 4, 8, 0), -1),        # no children
    ((64, 7, 3, 16, 4, 8, 0), -1),        # level bits not increasing
    ((64, 12, 3, 500, 4, 8, 0), -1),      # more generators than level 1 holds (448)
    ((8192, 26, 2, 16, 4, 8, 0), -2),     # wider than the library supports
])
def test_plan_create_rejects_bad_arguments_before_touching_the_gpu(lib, args, status):
    assert _create(lib, *args) == status


@pytest.mark.parametrize("d,level_bits,branching,active", [
    (5000, [13, 16], [0, 16], [4, 8]),                                    # d > 4096
    (64, [6, 19], [0, 16], [4, 8]),                                       # n_last > 3t (t = 6)
    (1024, [10, 14], [0, 64], [8, 300]),                                  # K_1 > 256
    (1024, [10, 14], [0, 5000], [1, 8]),                                  # Delta_1 > 4096
    (1024, [10, 15], [0, 256], [64, 32]),                                 # K_0 Delta_1 = 16384 candidates
    (1024, [10, 13, 16, 19, 22], [0, 32, 32, 32, 32], [256] * 5),        # k_tot = 1280 > 1024
])
def test_plans_outside_the_library_limits_are_unsupported(lib, d, level_bits, branching, active):
    """Valid hierarchies beyond the documented limits of dpb_plan_create_ex
    get DPB_EUNSUPPORTED, found on the host before any device call."""
    h = ctypes.c_void_p()
    st = lib.dpb_plan_create_ex(ctypes.byref(h), d, len(level_bits), binding._ints(level_bits),
                                binding._ints(branching), binding._ints(active), None, 0)
    assert st == -2


@pytest.mark.parametrize("d,level_bits,branching,active", [
    (1536, [11, 16], [0, 64], [2, 64]),
    (4096, [12, 16], [0, 16], [1, 16]),
    (2048, [11, 13, 15], [0, 16, 16], [4, 4, 8]),
])
def test_wide_rows_with_few_parents_are_within_the_limits(lib, d, level_bits, branching, active):
    """Hierarchies whose 16-column decode groups would not fit in LDS (d in
    the thousands, K_0 of 1 to 4) pass validation: the code kernels take
    fewer tokens per wave.  Without a GPU the call ends at the device upload
    (DPB_EHIP); with one it succeeds."""
    h = ctypes.c_void_p()
    st = lib.dpb_plan_create_ex(ctypes.byref(h), d, len(level_bits), binding._ints(level_bits),
                                binding._ints(branching), binding._ints(active), None, 0)
    if st == 0:
        lib.dpb_plan_destroy(h)
    assert st in (0, -3)


def test_compute_calls_reject_null_plan(lib):
    P = ctypes.c_void_p
    assert lib.dpb_encode(None, P(16), 0, 4, P(16), P(16), None, 0, None) == -1
    assert lib.dpb_decode(None, P(16), P(16), 4, P(16), 0, None) == -1
    assert lib.dpb_decode_bwd(None, P(16), P(16), 0, 4, P(16), P(16), 0, None) == -1
    assert lib.dpb_decode_bwd_ex(None, P(16), P(16), 0, 4, None, None, None, P(16), P(16), 0, None) == -1
    assert lib.dpb_encode_std(None, P(16), 0, 4, P(16), P(16), P(16), None, 0, None) == -1
    assert lib.dpb_plan_tables(None, P(16), P(16)) == -1
    assert lib.dpb_encode_workspace_bytes(None, 4) == 0
    assert lib.dpb_std_init(None, P(16), P(16), None) == -1
    assert lib.dpb_std_update(None, P(16), 0, 4, P(16), 0.1, 1e-6, P(16), P(16), P(16), 1 << 20, None) == -1
    assert lib.dpb_std_workspace_bytes(None) == 0
    assert lib.dpb_normalize(None, P(16), 0, P(16), 0, None, 4, 4, P(16), 0, None, None) == -1
    assert lib.dpb_normalize_bwd(None, P(16), 0, P(16), 0, P(16), 0, 4, P(32), 0, P(48), 0, 0, None) == -1
    assert lib.dpb_edit_codes(None, P(16), P(16), None, None, 4, P(16), P(32), P(48), 2, P(64), P(80), None) == -1
    assert lib.dpb_variance_loss(None, P(16), P(16), 4, 1, P(16), 1 << 20, P(16), None, None, None) == -1
    assert lib.dpb_variance_grad(None, 4, P(16), 1 << 20, P(16), None, None) == -1
    assert lib.dpb_variance_workspace_bytes(None, 4) == 0
    assert lib.dpb_plan_code_width(None) == 0
    lib.dpb_plan_destroy(None)


def test_create_ex_rejects_bad_generators(lib):
    h = ctypes.c_void_p()
    lb, br, ac = binding._ints([6, 9]), binding._ints([0, 2]), binding._ints([4, 4])
    dup = (ctypes.c_uint32 * 2)(100, 100)
    assert lib.dpb_plan_create_ex(ctypes.byref(h), 64, 2, lb, br, ac, dup, 0) == -1
    low = (ctypes.c_uint32 * 2)(63, 100)       # 63 lies in level 0
    assert lib.dpb_plan_create_ex(ctypes.byref(h), 64, 2, lb, br, ac, low, 0) == -1


def test_status_strings(lib):
    for s in (0, -1, -2, -3, -4):
        assert lib.dpb_status_string(s).startswith(b"DPB_")
