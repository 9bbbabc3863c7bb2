"""CPU oracle for the Deep Parity Bottleneck -- TEST INFRASTRUCTURE ONLY.

A plain, slow, fp64 implementation of what the paper defines (§2.1 parity
decoder, §2.2 parity encoder, App. A.4 seed matrix).  It is written in C
(`dpb_oracle.c`, built with gcc) and wrapped here with ctypes.  It shares no
code with the HIP library, and only the tests, the smoke check and the
benchmark's CPU-baseline leg may import it.

Functions whose parity against the paper cannot be pinned (they rest on a
reading of a point the paper leaves open) say "parity unpinned" below.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dpb_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with gcc -O2 -fopenmp into oracle/liboracle.so
    (again whenever the C source is newer than the library)."""
    stale = not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC)
    if force or stale:
        tmp = _LIB_PATH + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    lib = ctypes.CDLL(build())
    u32, i32, i64, u64, dbl = ctypes.c_uint32, ctypes.c_int, ctypes.c_int64, ctypes.c_uint64, ctypes.c_double
    P = ctypes.c_void_p
    sig = {
        "oracle_gf_mul": (u32, [u32, u32, i32, u32]),
        "oracle_gf_pow": (u32, [u32, u64, i32, u32]),
        "oracle_gf_inv": (u32, [u32, i32, u32]),
        "oracle_gf_trace": (u32, [u32, i32, u32]),
        "oracle_gf_order": (u32, [u32, i32, u32]),
        "oracle_poly_irreducible": (i32, [u64]),
        "oracle_pick_poly": (u32, [i32]),
        "oracle_primitive_element": (u32, [i32, u32]),
        "oracle_ceil_log2": (i32, [i32]),
        "oracle_masks": (i32, [i32, i32, P]),
        "oracle_phi": (dbl, [i32, P, i64, i32]),
        "oracle_generators": (i32, [i32, P, P, u64, P]),
        "oracle_splitmix64": (None, [u64, i32, P]),
        "oracle_scores": (None, [i32, P, P, i64, P, P]),
        "oracle_hierarchy": (i32, [i32, i32, i32, i32, i32, i32, P, P, P]),
        "oracle_encode": (i32, [i32, P, i32, P, P, P, P, P, i64, P, P, P, P]),
        "oracle_decode": (None, [i32, P, i32, P, P, i64, P]),
        "oracle_decode_bwd": (None, [i32, P, i32, P, P, i64, P, P]),
        "oracle_walsh_spectrum": (i32, [i32, P, i32, P]),
        "oracle_normalize": (None, [i32, i64, P, P, P, P]),
        "oracle_normalize_bwd": (None, [i32, i64, P, P, P, P, P]),
        "oracle_encode_std": (i32, [i32, P, i32, P, P, P, P, P, i64, P, P, P, P, P, P]),
        "oracle_std_update": (None, [i32, P, i32, P, P, P, P, P, i64, P, i32, dbl, P, P]),
        "oracle_std_r": (None, [i64, P, P, dbl, P]),
        "oracle_edit_codes": (None, [i64, i32, P, P, P, P, i64, P, P, P, P, P]),
        "oracle_variance_loss": (dbl, [i64, i32, P, P, i32, P]),
        "oracle_num_threads": (i32, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return ctypes.c_void_p(a.ctypes.data)


# ---------------------------------------------------------------- field

def gf_mul(a: int, b: int, t: int, poly: int) -> int:
    return int(_load().oracle_gf_mul(a, b, t, poly))


def gf_pow(a: int, e: int, t: int, poly: int) -> int:
    return int(_load().oracle_gf_pow(a, e, t, poly))


def gf_inv(a: int, t: int, poly: int) -> int:
    """xi^{-1} = xi^{2^t-2}, 0 -> 0 (App. A.4, inverse-by-exponentiation eq.)."""
    return int(_load().oracle_gf_inv(a, t, poly))


def gf_trace(y: int, t: int, poly: int) -> int:
    """Absolute trace (App. A.2)."""
    return int(_load().oracle_gf_trace(y, t, poly))


def gf_order(a: int, t: int, poly: int) -> int:
    return int(_load().oracle_gf_order(a, t, poly))


def poly_irreducible(f: int) -> bool:
    return bool(_load().oracle_poly_irreducible(f))


def pick_poly(t: int) -> int:
    """Modulus p(z) of degree t: fewest terms, then smallest value.

    Reproduces the paper's two choices (App. A.4); other degrees are a
    reading of the paper (parity unpinned for t not in {10, 11}).
    """
    return int(_load().oracle_pick_poly(t))


def primitive_element(t: int, poly: int) -> int:
    return int(_load().oracle_primitive_element(t, poly))


def ceil_log2(d: int) -> int:
    return int(_load().oracle_ceil_log2(d))


# ---------------------------------------------------------------- dictionary

def masks(d: int, r: int) -> np.ndarray:
    """Packed rows of the seed matrix M (App. A.4, parity-mask-row eq.).

    d = 2^t follows the paper exactly.  d not a power of two and r > 2t are
    readings (parity unpinned against the paper).
    """
    out = np.zeros(d, dtype=np.uint32)
    t = _load().oracle_masks(d, r, _ptr(out))
    if t < 0:
        raise ValueError(f"oracle_masks: unsupported d={d}, r={r}")
    return out


def phi(d: int, m: np.ndarray, i: int) -> np.ndarray:
    """Direction phi_i (§2.1 Eqs. 1-2) as an fp64 vector, one entry at a time."""
    lib = _load()
    return np.array([lib.oracle_phi(d, _ptr(m), int(i), k) for k in range(d)], dtype=np.float64)


def generators(nbits: Sequence[int], delta: Sequence[int], seed: int = 0) -> list[np.ndarray]:
    """Per-level generator sets (§2.2; sampling rule is a reading, parity unpinned)."""
    L = len(nbits)
    nb = np.asarray(nbits, dtype=np.int32)
    dl = np.asarray(delta, dtype=np.int32)
    total = int(dl[1:].sum()) if L > 1 else 0
    out = np.zeros(max(total, 1), dtype=np.uint32)
    rc = _load().oracle_generators(L, _ptr(nb), _ptr(dl), seed & (2**64 - 1), _ptr(out))
    if rc < 0:
        raise ValueError("oracle_generators: level too small for its branching")
    res, off = [np.zeros(0, dtype=np.uint32)], 0
    for l in range(1, L):
        res.append(out[off:off + dl[l]].copy())
        off += int(dl[l])
    return res


def splitmix64(state: int, n: int) -> list[int]:
    """The first n outputs of the SplitMix64 generator (Steele, Lea and Flood
    2014) from `state`, the stream the generator sampling draws from."""
    out = np.zeros(max(n, 1), dtype=np.uint64)
    _load().oracle_splitmix64(state & (2**64 - 1), n, _ptr(out))
    return [int(v) for v in out[:n]]


def hierarchy(d: int, n: int, levels: int, branching: int, beam: int, k: int):
    """Config terms -> (n_l, Delta_l, K_l) (reading of App. G Table 6; parity unpinned)."""
    nb = np.zeros(levels, dtype=np.int32)
    dl = np.zeros(levels, dtype=np.int32)
    ac = np.zeros(levels, dtype=np.int32)
    if _load().oracle_hierarchy(d, n, levels, branching, beam, k, _ptr(nb), _ptr(dl), _ptr(ac)) < 0:
        raise ValueError("oracle_hierarchy: bad arguments")
    return nb.tolist(), dl.tolist(), ac.tolist()


# ---------------------------------------------------------------- the path

def encode(d: int, m: np.ndarray, nbits, active, delta, gens: list[np.ndarray], x: np.ndarray):
    """Beam-search encoder (§2.2).  x: [T, d] (any float dtype; used as fp64).

    Returns idx [T, k_tot] int32, coef [T, k_tot] fp64, and the boundary and
    order margins [T, L] used to exempt near-ties when comparing with a
    finite-precision implementation.
    """
    x = np.ascontiguousarray(x, dtype=np.float64)
    T = x.shape[0]
    assert x.shape[1] == d
    L = len(nbits)
    nb = np.asarray(nbits, dtype=np.int32)
    ac = np.asarray(active, dtype=np.int32)
    dl = np.asarray(delta, dtype=np.int32)
    g = np.concatenate([np.asarray(gg, dtype=np.uint32) for gg in gens[1:]]) if L > 1 else np.zeros(1, np.uint32)
    g = np.ascontiguousarray(g if g.size else np.zeros(1, np.uint32), dtype=np.uint32)
    k_tot = int(ac.sum())
    idx = np.zeros((T, k_tot), dtype=np.int32)
    coef = np.zeros((T, k_tot), dtype=np.float64)
    margin = np.zeros((T, L), dtype=np.float64)
    order = np.zeros((T, L), dtype=np.float64)
    rc = _load().oracle_encode(d, _ptr(m), L, _ptr(nb), _ptr(ac), _ptr(dl), _ptr(g), _ptr(x), T,
                               _ptr(idx), _ptr(coef), _ptr(margin), _ptr(order))
    if rc < 0:
        raise ValueError("oracle_encode: bad arguments")
    return idx, coef, margin, order


def scores(d: int, m: np.ndarray, x_row: np.ndarray, ids) -> np.ndarray:
    """<phi_c, x> in fp64 for each feature c of ids (basis features give the
    coordinate itself), x_row one activation row [d]."""
    x_row = np.ascontiguousarray(x_row, dtype=np.float64)
    assert x_row.shape == (d,)
    ids = np.ascontiguousarray(np.asarray(ids, dtype=np.int64).reshape(-1))
    out = np.zeros(max(ids.size, 1), dtype=np.float64)
    if ids.size:
        _load().oracle_scores(d, _ptr(m), _ptr(x_row), ids.size, _ptr(ids), _ptr(out))
    return out[: ids.size]


def _hier_arrays(nbits, active, delta, gens):
    L = len(nbits)
    nb = np.asarray(nbits, dtype=np.int32)
    ac = np.asarray(active, dtype=np.int32)
    dl = np.asarray(delta, dtype=np.int32)
    g = np.concatenate([np.asarray(gg, dtype=np.uint32) for gg in gens[1:]]) if L > 1 else np.zeros(1, np.uint32)
    g = np.ascontiguousarray(g if g.size else np.zeros(1, np.uint32), dtype=np.uint32)
    return L, nb, ac, dl, g


def encode_std(d: int, m: np.ndarray, nbits, active, delta, gens: list[np.ndarray], x: np.ndarray,
               mu: np.ndarray, r: np.ndarray):
    """Beam-search encoder on standardized scores z = (s - mu) r (§2.2 "Score
    Standardization"); mu and r are fp32 per feature (2^n_last entries each).
    Level-0 z is taken in fp32, the levels above in fp64.  Returns idx, coef
    (= z), and the margins of |z| as in encode()."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    T = x.shape[0]
    assert x.shape[1] == d
    L, nb, ac, dl, g = _hier_arrays(nbits, active, delta, gens)
    mu = np.ascontiguousarray(mu, dtype=np.float32)
    r = np.ascontiguousarray(r, dtype=np.float32)
    assert mu.shape == r.shape == (1 << int(nb[-1]),)
    k_tot = int(ac.sum())
    idx = np.zeros((T, k_tot), dtype=np.int32)
    coef = np.zeros((T, k_tot), dtype=np.float64)
    margin = np.zeros((T, L), dtype=np.float64)
    order = np.zeros((T, L), dtype=np.float64)
    rc = _load().oracle_encode_std(d, _ptr(m), L, _ptr(nb), _ptr(ac), _ptr(dl), _ptr(g), _ptr(x), T,
                                   _ptr(mu), _ptr(r), _ptr(idx), _ptr(coef), _ptr(margin), _ptr(order))
    if rc < 0:
        raise ValueError("oracle_encode_std: bad arguments")
    return idx, coef, margin, order


def std_update(d: int, m: np.ndarray, nbits, active, delta, gens: list[np.ndarray], x: np.ndarray,
               idx: np.ndarray, mu: np.ndarray, m2: np.ndarray, beta: float, sample: int = 64):
    """EMA update of the standardization statistics after a batch (§2.2
    "Score Standardization"; the sample and the moving raw moments are
    readings): mu and m2 are the moving first and second raw moments of each
    feature's score while it is a candidate.  x is the batch, idx its code;
    mu, m2 fp64 [2^n_last].  Returns updated copies (mu, m2)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    T = x.shape[0]
    L, nb, ac, dl, g = _hier_arrays(nbits, active, delta, gens)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    assert idx.shape == (T, int(ac.sum()))
    mu = np.array(mu, dtype=np.float64, order="C")
    m2 = np.array(m2, dtype=np.float64, order="C")
    assert mu.shape == m2.shape == (1 << int(nb[-1]),)
    _load().oracle_std_update(d, _ptr(m), L, _ptr(nb), _ptr(ac), _ptr(dl), _ptr(g), _ptr(x), T, _ptr(idx),
                              int(sample), float(beta), _ptr(mu), _ptr(m2))
    return mu, m2


def std_r(mu: np.ndarray, m2: np.ndarray, eps: float) -> np.ndarray:
    """r = 1 / sqrt(max(m2 - mu^2, 0) + eps): the inverse standard deviation
    the two moving moments imply, fp64."""
    mu = np.ascontiguousarray(mu, dtype=np.float64)
    m2 = np.ascontiguousarray(m2, dtype=np.float64)
    assert mu.shape == m2.shape and mu.ndim == 1
    r = np.zeros_like(mu)
    _load().oracle_std_r(mu.shape[0], _ptr(mu), _ptr(m2), float(eps), _ptr(r))
    return r


def decode(d: int, m: np.ndarray, idx: np.ndarray, coef: np.ndarray) -> np.ndarray:
    """x_hat = sum_i a_i phi_i (§2.1), fp64.  idx < 0 slots are padding."""
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    coef = np.ascontiguousarray(coef, dtype=np.float64)
    T, k = idx.shape
    y = np.zeros((T, d), dtype=np.float64)
    _load().oracle_decode(d, _ptr(m), k, _ptr(idx), _ptr(coef), T, _ptr(y))
    return y


def decode_bwd(d: int, m: np.ndarray, idx: np.ndarray, g: np.ndarray):
    """grad_coef = Phi_S^T g and grad_x = Phi_S grad_coef, fp64."""
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    g = np.ascontiguousarray(g, dtype=np.float64)
    T, k = idx.shape
    gc = np.zeros((T, k), dtype=np.float64)
    gx = np.zeros((T, d), dtype=np.float64)
    _load().oracle_decode_bwd(d, _ptr(m), k, _ptr(idx), _ptr(g), T, _ptr(gc), _ptr(gx))
    return gc, gx


def normalize(u: np.ndarray, ref: np.ndarray):
    """Normalized reconstruction (§2.2): y = u ||ref|| / ||u|| per row (0 when
    ||u|| = 0), fp64.  Returns y and norms [T, 2] = (||ref||, ||u||)."""
    u = np.ascontiguousarray(u, dtype=np.float64)
    ref = np.ascontiguousarray(ref, dtype=np.float64)
    T, d = u.shape
    y = np.zeros_like(u)
    norms = np.zeros((T, 2), dtype=np.float64)
    _load().oracle_normalize(d, T, _ptr(u), _ptr(ref), _ptr(y), _ptr(norms))
    return y, norms


def normalize_bwd(g: np.ndarray, u: np.ndarray, ref: np.ndarray):
    """Backward of `normalize` for dL/dy = g: returns (dL/du, dL/dref), fp64."""
    g = np.ascontiguousarray(g, dtype=np.float64)
    u = np.ascontiguousarray(u, dtype=np.float64)
    ref = np.ascontiguousarray(ref, dtype=np.float64)
    T, d = u.shape
    gu = np.zeros_like(u)
    gr = np.zeros_like(u)
    _load().oracle_normalize_bwd(d, T, _ptr(g), _ptr(u), _ptr(ref), _ptr(gu), _ptr(gr))
    return gu, gr


def edit_codes(idx: np.ndarray, coef: np.ndarray, tidx: np.ndarray, tcoef: np.ndarray, edits):
    """Edit candidates of the greedy feature editing (App. C.3).

    idx/coef is the source code [T, k], tidx/tcoef the target code of the same
    shape; edits is a list of (row, slot, op).  Output row e is source row
    `row` with slot `slot` edited: op 0 zero the coefficient, 1 replace index
    and coefficient by the target's at that position, 2 rescale (take the
    target's coefficient, keep the index), 3 no change.  Out-of-range edits
    give an all-padding row.  Returns (idx int32 [E, k], coef fp64 [E, k])."""
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    coef = np.ascontiguousarray(coef, dtype=np.float64)
    tidx = np.ascontiguousarray(tidx, dtype=np.int32)
    tcoef = np.ascontiguousarray(tcoef, dtype=np.float64)
    T, k = idx.shape
    assert tidx.shape == (T, k) and tcoef.shape == (T, k)
    E = len(edits)
    rows = np.array([e[0] for e in edits] or [0], dtype=np.int32)
    slots = np.array([e[1] for e in edits] or [0], dtype=np.int32)
    ops = np.array([e[2] for e in edits] or [0], dtype=np.int32)
    out_idx = np.zeros((max(E, 1), k), dtype=np.int32)
    out_coef = np.zeros((max(E, 1), k), dtype=np.float64)
    _load().oracle_edit_codes(T, k, _ptr(idx), _ptr(coef), _ptr(tidx), _ptr(tcoef), E, _ptr(rows), _ptr(slots),
                              _ptr(ops), _ptr(out_idx), _ptr(out_coef))
    return out_idx[:E], out_coef[:E]


def variance_loss(idx: np.ndarray, coef: np.ndarray, n_min: int):
    """Variance auxiliary loss (§2.2) and its gradient with respect to coef.

    Population variance per feature over the slots holding it; features with
    fewer than n_min samples are left out (the variance estimator and the
    treatment of a feature repeated within one token are readings).
    """
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    coef = np.ascontiguousarray(coef, dtype=np.float64)
    T, k = idx.shape
    grad = np.zeros((T, k), dtype=np.float64)
    loss = _load().oracle_variance_loss(T, k, _ptr(idx), _ptr(coef), int(n_min), _ptr(grad))
    return float(loss), grad


def layer_backward(d: int, m: np.ndarray, idx: np.ndarray, coef: np.ndarray, x: np.ndarray, gy: np.ndarray,
                   gloss: float, n_min: int, normalized: bool = True, r_slot: np.ndarray | None = None):
    """Gradients of a DPB layer with the indices held fixed (coef = Phi_S x,
    or with standardization coef = (Phi_S x - mu) r; u = Phi_S^T coef,
    y = u ||x|| / ||u|| when normalized, else y = u) under the loss
    <gy, y> + gloss * L_var(coef), composed from the oracle's parts:
        gu, gref  = normalize_bwd(gy, u, x)            (gu = gy, gref = 0 if not normalized)
        grad_coef = Phi_S^T gu + gloss * dL_var/dcoef
        grad_x    = Phi_S (r grad_coef) + gref         (r = r_slot [T, k], else 1)
    Returns (grad_coef [T, k], grad_x [T, d]) in fp64."""
    x = np.asarray(x, dtype=np.float64)
    gy = np.asarray(gy, dtype=np.float64)
    u = decode(d, m, idx, coef)
    if normalized:
        gu, gref = normalize_bwd(gy, u, x)
    else:
        gu, gref = gy, np.zeros_like(x)
    gc, _ = decode_bwd(d, m, idx, gu)
    _, vg = variance_loss(idx, coef, n_min)
    gc = gc + gloss * vg
    scaled = gc if r_slot is None else gc * np.asarray(r_slot, dtype=np.float64)
    return gc, decode(d, m, idx, scaled) + gref


def num_threads() -> int:
    """OpenMP threads the oracle's token loops run on."""
    return int(_load().oracle_num_threads())


def walsh_spectrum(d: int, m: np.ndarray, r: int) -> np.ndarray:
    """S(u) = sum_iota (-1)^{popcount(M_iota & u)}, all u < 2^r, via one FWHT."""
    S = np.zeros(1 << r, dtype=np.int64)
    if _load().oracle_walsh_spectrum(d, _ptr(m), r, _ptr(S)) < 0:
        raise ValueError("oracle_walsh_spectrum: r out of range")
    return S
