"""ctypes binding over libdpb.so (the C ABI in include/dpb.h).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  torch supplies device memory and the current stream.  There is no
fallback: if libdpb.so is missing the first call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
lib_path = os.path.join(_HERE, "libdpb.so")

DPB_F32, DPB_BF16 = 0, 1
_STATUS = {0: "DPB_OK", -1: "DPB_EINVAL", -2: "DPB_EUNSUPPORTED", -3: "DPB_EHIP", -4: "DPB_ENOMEM"}
MAX_LEVELS = 8

_lib = None


class DPBError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} failed: {_STATUS.get(status, status)}")


def load():
    """Loads libdpb.so (built by `python -m paper_2607_20652_amd.build`)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(lib_path):
        raise RuntimeError(f"{lib_path} is not built; run `python -m paper_2607_20652_amd.build`")
    lib = ctypes.CDLL(lib_path)
    i32, i64, u64, P = ctypes.c_int, ctypes.c_int64, ctypes.c_uint64, ctypes.c_void_p
    sig = {
        "dpb_status_string": (ctypes.c_char_p, [i32]),
        "dpb_hierarchy": (i32, [i32, i32, i32, i32, i32, i32, P, P, P]),
        "dpb_build_tables": (i32, [i32, i32, P, P, u64, P, P]),
        "dpb_plan_create": (i32, [P, i32, i32, i32, i32, i32, i32, u64]),
        "dpb_plan_create_ex": (i32, [P, i32, i32, P, P, P, P, u64]),
        "dpb_plan_destroy": (None, [P]),
        "dpb_plan_code_width": (i32, [P]),
        "dpb_plan_describe": (i32, [P, P, P, P, P, P, P, P]),
        "dpb_encode": (i32, [P, P, i32, i64, P, P, P]),
        "dpb_decode": (i32, [P, P, P, i64, P, i32, P]),
        "dpb_decode_bwd": (i32, [P, P, P, i32, i64, P, P, i32, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(fn: str, status: int):
    if status != 0:
        raise DPBError(fn, status)


def _ints(vals: Sequence[int]):
    arr = (ctypes.c_int * MAX_LEVELS)()
    for i, v in enumerate(vals):
        arr[i] = int(v)
    return arr


def hierarchy(d: int, n_bits: int, levels: int, branching: int, beam: int, k: int):
    """(level_bits, branching, active) the library derives from configuration terms."""
    nb, br, ac = _ints([]), _ints([]), _ints([])
    _check("dpb_hierarchy", load().dpb_hierarchy(d, n_bits, levels, branching, beam, k, nb, br, ac))
    return list(nb[:levels]), list(br[:levels]), list(ac[:levels])


def build_tables(d: int, level_bits: Sequence[int], branching: Sequence[int], seed: int = 0):
    """Host-only tables (masks [d], generators [sum Delta]) as Python int lists."""
    L = len(level_bits)
    masks = (ctypes.c_uint32 * d)()
    ng = max(1, sum(int(b) for b in list(branching)[1:]))
    gens = (ctypes.c_uint32 * ng)()
    _check("dpb_build_tables",
           load().dpb_build_tables(d, L, _ints(level_bits), _ints(branching), seed & (2**64 - 1), masks, gens))
    return list(masks), list(gens[: sum(int(b) for b in list(branching)[1:])])


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return DPB_F32
    if t.dtype == torch.bfloat16:
        return DPB_BF16
    raise TypeError(f"unsupported dtype {t.dtype}; use float32 or bfloat16")


def _stream(t: torch.Tensor):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _dev(t: torch.Tensor, name: str):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


class Plan:
    """A DPB hierarchy and its device tables (one plan per device)."""

    def __init__(self, d: int, n_bits: int | None = None, levels: int | None = None, branching: int | None = None,
                 beam: int | None = None, k: int | None = None, seed: int = 0, *,
                 level_bits: Sequence[int] | None = None, branchings: Sequence[int] | None = None,
                 active: Sequence[int] | None = None, generators: Sequence[int] | None = None,
                 device: torch.device | int | None = None):
        lib = load()
        self._handle = ctypes.c_void_p()
        dev = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device("cuda", device) \
            if isinstance(device, int) else torch.device(device)
        self.device = dev
        with torch.cuda.device(dev):
            if level_bits is None:
                st = lib.dpb_plan_create(ctypes.byref(self._handle), d, n_bits, levels, branching, beam, k,
                                         seed & (2**64 - 1))
                _check("dpb_plan_create", st)
            else:
                L = len(level_bits)
                g = None
                if generators is not None:
                    g = (ctypes.c_uint32 * max(1, len(generators)))(*[int(v) for v in generators])
                st = lib.dpb_plan_create_ex(ctypes.byref(self._handle), d, L, _ints(level_bits),
                                            _ints(branchings if branchings is not None else [0] * L),
                                            _ints(active), g, seed & (2**64 - 1))
                _check("dpb_plan_create_ex", st)
        self.d = d
        nb, br, ac = _ints([]), _ints([]), _ints([])
        dd, ll = ctypes.c_int(), ctypes.c_int()
        _check("dpb_plan_describe", lib.dpb_plan_describe(self._handle, ctypes.byref(dd), ctypes.byref(ll), nb, br,
                                                          ac, None, None))
        self.levels = ll.value
        self.level_bits = list(nb[: self.levels])
        self.branching = list(br[: self.levels])
        self.active = list(ac[: self.levels])
        self.k_tot = lib.dpb_plan_code_width(self._handle)

    def tables(self):
        """Host copies of the plan's masks [d] and generators (level by level)."""
        lib = load()
        masks = (ctypes.c_uint32 * self.d)()
        ng = max(1, sum(self.branching[1:]))
        gens = (ctypes.c_uint32 * ng)()
        _check("dpb_plan_describe", lib.dpb_plan_describe(self._handle, None, None, None, None, None, masks, gens))
        return list(masks), list(gens[: sum(self.branching[1:])])

    def close(self):
        if getattr(self, "_handle", None) and self._handle.value:
            load().dpb_plan_destroy(self._handle)
            self._handle = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def encode(plan: Plan, x: torch.Tensor, idx: torch.Tensor | None = None, coef: torch.Tensor | None = None):
    """x [T, d] fp32/bf16 (device) -> (idx [T, k_tot] int32, coef [T, k_tot] fp32)."""
    T = x.shape[0]
    assert x.dim() == 2 and x.shape[1] == plan.d
    if idx is None:
        idx = torch.empty((T, plan.k_tot), dtype=torch.int32, device=x.device)
    if coef is None:
        coef = torch.empty((T, plan.k_tot), dtype=torch.float32, device=x.device)
    _check("dpb_encode", load().dpb_encode(plan._handle, _dev(x, "x"), _dtype_code(x), T, _dev(idx, "idx"),
                                           _dev(coef, "coef"), _stream(x)))
    return idx, coef


def decode(plan: Plan, idx: torch.Tensor, coef: torch.Tensor, out_dtype: torch.dtype = torch.float32,
           y: torch.Tensor | None = None):
    """(idx, coef) [T, k_tot] -> y [T, d] in out_dtype (fp32 or bf16)."""
    T = idx.shape[0]
    assert idx.dtype == torch.int32 and coef.dtype == torch.float32 and idx.shape == coef.shape
    assert idx.shape[1] == plan.k_tot
    if y is None:
        y = torch.empty((T, plan.d), dtype=out_dtype, device=idx.device)
    _check("dpb_decode", load().dpb_decode(plan._handle, _dev(idx, "idx"), _dev(coef, "coef"), T, _dev(y, "y"),
                                           _dtype_code(y), _stream(idx)))
    return y


def decode_bwd(plan: Plan, idx: torch.Tensor, grad_y: torch.Tensor, gx_dtype: torch.dtype | None = None,
               grad_coef: torch.Tensor | None = None, grad_x: torch.Tensor | None = None):
    """(idx [T, k_tot], grad_y [T, d]) -> (grad_coef [T, k_tot] fp32, grad_x [T, d])."""
    T = idx.shape[0]
    assert idx.dtype == torch.int32 and idx.shape[1] == plan.k_tot and grad_y.shape == (T, plan.d)
    if grad_coef is None:
        grad_coef = torch.empty((T, plan.k_tot), dtype=torch.float32, device=idx.device)
    if grad_x is None:
        grad_x = torch.empty((T, plan.d), dtype=gx_dtype or grad_y.dtype, device=idx.device)
    _check("dpb_decode_bwd", load().dpb_decode_bwd(plan._handle, _dev(idx, "idx"), _dev(grad_y, "grad_y"),
                                                   _dtype_code(grad_y), T, _dev(grad_coef, "grad_coef"),
                                                   _dev(grad_x, "grad_x"), _dtype_code(grad_x), _stream(idx)))
    return grad_coef, grad_x


def forward(plan: Plan, x: torch.Tensor, out_dtype: torch.dtype | None = None):
    """encode then decode: x -> (idx, coef, y)."""
    idx, coef = encode(plan, x)
    return idx, coef, decode(plan, idx, coef, out_dtype or x.dtype)
