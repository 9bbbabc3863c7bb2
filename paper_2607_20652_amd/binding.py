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
EDIT_ZERO, EDIT_REPLACE, EDIT_RESCALE, EDIT_NONE = 0, 1, 2, 3
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
        "dpb_plan_tables": (i32, [P, P, P]),
        "dpb_encode": (i32, [P, P, i32, i64, P, P, P, ctypes.c_size_t, P]),
        "dpb_decode": (i32, [P, P, P, i64, P, i32, P]),
        "dpb_forward": (i32, [P, P, i32, i64, P, P, P, P, i32, P, ctypes.c_size_t, P]),
        "dpb_decode_bwd": (i32, [P, P, P, i32, i64, P, P, i32, P]),
        "dpb_decode_bwd_ex": (i32, [P, P, P, i32, i64, P, P, P, P, P, i32, P]),
        "dpb_encode_std": (i32, [P, P, i32, i64, P, P, P, P, ctypes.c_size_t, P]),
        "dpb_encode_noalloc": (i32, [P, P, i32, i64, P, P, P, P]),
        "dpb_encode_workspace_bytes": (ctypes.c_size_t, [P, i64]),
        "dpb_std_init": (i32, [P, P, P, P]),
        "dpb_std_workspace_bytes": (ctypes.c_size_t, [P]),
        "dpb_std_update": (i32, [P, P, i32, i64, P, ctypes.c_float, ctypes.c_float, P, P, P, ctypes.c_size_t, P]),
        "dpb_normalize": (i32, [P, P, i32, P, i32, P, i64, i64, P, i32, P, P]),
        "dpb_normalize_bwd": (i32, [P, P, i32, P, i32, P, i32, i64, P, i32, P, i32, i32, P]),
        "dpb_edit_codes": (i32, [P, P, P, P, P, i64, P, P, P, i64, P, P, P]),
        "dpb_variance_workspace_bytes": (ctypes.c_size_t, [P, i64]),
        "dpb_variance_loss": (i32, [P, P, P, i64, i32, P, ctypes.c_size_t, P, P, P, P]),
        "dpb_variance_grad": (i32, [P, i64, P, ctypes.c_size_t, P, P, P]),
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
        _check("dpb_plan_tables", lib.dpb_plan_tables(self._handle, masks, gens))
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


def encode_workspace(plan: Plan, T: int, device) -> torch.Tensor | None:
    """Workspace for encode of T tokens, or None when the plan needs none."""
    n = int(load().dpb_encode_workspace_bytes(plan._handle, int(T)))
    return None if n == 0 else torch.empty(((n + 15) // 16) * 4, dtype=torch.float32, device=device)


def encode(plan: Plan, x: torch.Tensor, idx: torch.Tensor | None = None, coef: torch.Tensor | None = None,
           stats: torch.Tensor | None = None, workspace: torch.Tensor | None = None):
    """x [T, d] fp32/bf16 (device) -> (idx [T, k_tot] int32, coef [T, k_tot] fp32); on
    standardized scores when stats is given.  A workspace is allocated when the
    plan needs one (wide hierarchies) and none is given."""
    T = x.shape[0]
    assert x.dim() == 2 and x.shape[1] == plan.d
    if idx is None:
        idx = torch.empty((T, plan.k_tot), dtype=torch.int32, device=x.device)
    if coef is None:
        coef = torch.empty((T, plan.k_tot), dtype=torch.float32, device=x.device)
    if workspace is None:
        workspace = encode_workspace(plan, T, x.device)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    if stats is None:
        _check("dpb_encode", load().dpb_encode(plan._handle, _dev(x, "x"), _dtype_code(x), T, _dev(idx, "idx"),
                                               _dev(coef, "coef"), _opt(workspace, "workspace"), nbytes,
                                               _stream(x)))
    else:
        _check("dpb_encode_std", load().dpb_encode_std(plan._handle, _dev(x, "x"), _dtype_code(x), T,
                                                       _dev(stats, "stats"), _dev(idx, "idx"), _dev(coef, "coef"),
                                                       _opt(workspace, "workspace"), nbytes, _stream(x)))
    return idx, coef


def encode_noalloc(plan: Plan, x: torch.Tensor, idx: torch.Tensor, coef: torch.Tensor,
                   stats: torch.Tensor | None = None):
    """encode (stats None) or encode_std into the given idx, coef [T, k_tot]
    through the library's allocation-free entry point (no workspace)."""
    T = x.shape[0]
    assert x.dim() == 2 and x.shape[1] == plan.d and idx.shape == coef.shape == (T, plan.k_tot)
    _check("dpb_encode_noalloc", load().dpb_encode_noalloc(plan._handle, _dev(x, "x"), _dtype_code(x), T,
                                                           _opt(stats, "stats"), _dev(idx, "idx"),
                                                           _dev(coef, "coef"), _stream(x)))
    return idx, coef


def forward(plan: Plan, x: torch.Tensor, idx: torch.Tensor | None = None, coef: torch.Tensor | None = None,
            y: torch.Tensor | None = None, stats: torch.Tensor | None = None, out_dtype: torch.dtype | None = None,
            workspace: torch.Tensor | None = None):
    """x [T, d] -> (idx, coef, y): encode (on standardized scores when stats is
    given) and decode in one library call (dpb_forward); y [T, d] in out_dtype
    (default: the type of x)."""
    T = x.shape[0]
    assert x.dim() == 2 and x.shape[1] == plan.d
    if idx is None:
        idx = torch.empty((T, plan.k_tot), dtype=torch.int32, device=x.device)
    if coef is None:
        coef = torch.empty((T, plan.k_tot), dtype=torch.float32, device=x.device)
    if y is None:
        y = torch.empty((T, plan.d), dtype=out_dtype or x.dtype, device=x.device)
    if workspace is None:
        workspace = encode_workspace(plan, T, x.device)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check("dpb_forward", load().dpb_forward(plan._handle, _dev(x, "x"), _dtype_code(x), T, _opt(stats, "stats"),
                                             _dev(idx, "idx"), _dev(coef, "coef"), _dev(y, "y"), _dtype_code(y),
                                             _opt(workspace, "workspace"), nbytes, _stream(x)))
    return idx, coef, y


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


def _opt(t: torch.Tensor | None, name: str):
    return None if t is None else _dev(t, name)


def decode_bwd_ex(plan: Plan, idx: torch.Tensor, grad_y: torch.Tensor, add_grad_coef: torch.Tensor | None = None,
                  add_grad_x: torch.Tensor | None = None, gx_dtype: torch.dtype | None = None,
                  grad_coef: torch.Tensor | None = None, grad_x: torch.Tensor | None = None,
                  stats: torch.Tensor | None = None):
    """decode_bwd plus extra terms: grad_coef = Phi^T g + add_grad_coef,
    grad_x = Phi (r * grad_coef) + add_grad_x, r from the standardization
    statistics when given (else 1); add_grad_x is in grad_x's dtype and may
    be grad_x itself."""
    T = idx.shape[0]
    assert idx.dtype == torch.int32 and idx.shape[1] == plan.k_tot and grad_y.shape == (T, plan.d)
    if grad_coef is None:
        grad_coef = torch.empty((T, plan.k_tot), dtype=torch.float32, device=idx.device)
    if grad_x is None:
        grad_x = torch.empty((T, plan.d), dtype=gx_dtype or grad_y.dtype, device=idx.device)
    if add_grad_coef is not None:
        assert add_grad_coef.dtype == torch.float32 and add_grad_coef.shape == (T, plan.k_tot)
    if add_grad_x is not None:
        assert add_grad_x.dtype == grad_x.dtype and add_grad_x.shape == (T, plan.d)
    _check("dpb_decode_bwd_ex", load().dpb_decode_bwd_ex(
        plan._handle, _dev(idx, "idx"), _dev(grad_y, "grad_y"), _dtype_code(grad_y), T,
        _opt(add_grad_coef, "add_grad_coef"), _opt(add_grad_x, "add_grad_x"), _opt(stats, "stats"),
        _dev(grad_coef, "grad_coef"), _dev(grad_x, "grad_x"), _dtype_code(grad_x), _stream(idx)))
    return grad_coef, grad_x


def normalize(plan: Plan, u: torch.Tensor, ref: torch.Tensor, ref_rows: torch.Tensor | None = None,
              out_dtype: torch.dtype | None = None, y: torch.Tensor | None = None, with_norms: bool = False):
    """y = u ||ref_r|| / ||u|| per row (r = ref_rows[t] or t); optionally the
    (||ref_r||, ||u||) pairs [T, 2]."""
    T = u.shape[0]
    assert u.shape == (T, plan.d) and ref.dim() == 2 and ref.shape[1] == plan.d
    if ref_rows is not None:
        assert ref_rows.dtype == torch.int32 and ref_rows.shape == (T,)
    else:
        assert ref.shape[0] == T
    if y is None:
        y = torch.empty((T, plan.d), dtype=out_dtype or u.dtype, device=u.device)
    norms = torch.empty((T, 2), dtype=torch.float32, device=u.device) if with_norms else None
    _check("dpb_normalize", load().dpb_normalize(
        plan._handle, _dev(u, "u"), _dtype_code(u), _dev(ref, "ref"), _dtype_code(ref), _opt(ref_rows, "ref_rows"),
        ref.shape[0], T, _dev(y, "y"), _dtype_code(y), _opt(norms, "norms"), _stream(u)))
    return (y, norms) if with_norms else y


def normalize_bwd(plan: Plan, g: torch.Tensor, u: torch.Tensor, ref: torch.Tensor,
                  gu_dtype: torch.dtype | None = None, grad_ref: torch.Tensor | None = None,
                  accumulate: bool = False, gr_dtype: torch.dtype | None = None):
    """(grad_u, grad_ref) of normalize for upstream g; grad_ref is added to
    the given buffer when accumulate is True."""
    T = u.shape[0]
    assert g.shape == u.shape == ref.shape == (T, plan.d)
    grad_u = torch.empty((T, plan.d), dtype=gu_dtype or g.dtype, device=u.device)
    if grad_ref is None:
        assert not accumulate
        grad_ref = torch.empty((T, plan.d), dtype=gr_dtype or ref.dtype, device=u.device)
    _check("dpb_normalize_bwd", load().dpb_normalize_bwd(
        plan._handle, _dev(g, "g"), _dtype_code(g), _dev(u, "u"), _dtype_code(u), _dev(ref, "ref"),
        _dtype_code(ref), T, _dev(grad_u, "grad_u"), _dtype_code(grad_u), _dev(grad_ref, "grad_ref"),
        _dtype_code(grad_ref), int(bool(accumulate)), _stream(u)))
    return grad_u, grad_ref


def edit_codes(plan: Plan, idx: torch.Tensor, coef: torch.Tensor, rows: torch.Tensor, slots: torch.Tensor,
               ops: torch.Tensor, tgt_idx: torch.Tensor | None = None, tgt_coef: torch.Tensor | None = None):
    """One edited copy of source row rows[e] per edit (slot slots[e], op
    ops[e]: EDIT_ZERO, EDIT_REPLACE, EDIT_RESCALE, EDIT_NONE) -> (idx, coef) [E, k_tot]."""
    T, E = idx.shape[0], rows.shape[0]
    assert idx.shape == coef.shape == (T, plan.k_tot) and idx.dtype == torch.int32 and coef.dtype == torch.float32
    for t in (rows, slots, ops):
        assert t.dtype == torch.int32 and t.shape == (E,)
    out_idx = torch.empty((E, plan.k_tot), dtype=torch.int32, device=idx.device)
    out_coef = torch.empty((E, plan.k_tot), dtype=torch.float32, device=idx.device)
    _check("dpb_edit_codes", load().dpb_edit_codes(
        plan._handle, _dev(idx, "idx"), _dev(coef, "coef"), _opt(tgt_idx, "tgt_idx"), _opt(tgt_coef, "tgt_coef"), T,
        _dev(rows, "rows"), _dev(slots, "slots"), _dev(ops, "ops"), E, _dev(out_idx, "out_idx"),
        _dev(out_coef, "out_coef"), _stream(idx)))
    return out_idx, out_coef


def variance_workspace_bytes(plan: Plan, T: int) -> int:
    return int(load().dpb_variance_workspace_bytes(plan._handle, int(T)))


def variance_workspace(plan: Plan, T: int, device) -> torch.Tensor:
    """A device buffer of dpb_variance_workspace_bytes(plan, T) bytes."""
    return torch.empty((variance_workspace_bytes(plan, T) + 15) // 16 * 4, dtype=torch.float32, device=device)


def variance_loss(plan: Plan, idx: torch.Tensor, coef: torch.Tensor, n_min: int, with_grad: bool = True,
                  workspace: torch.Tensor | None = None, grad_scale: torch.Tensor | None = None):
    """Variance auxiliary loss of a batch of codes -> (loss [] fp32, grad_coef
    [T, k_tot] fp32 or None); grad_coef is multiplied by the device scalar
    grad_scale when given."""
    T = idx.shape[0]
    assert idx.shape == coef.shape == (T, plan.k_tot) and idx.dtype == torch.int32 and coef.dtype == torch.float32
    if workspace is None:
        workspace = variance_workspace(plan, T, idx.device)
    loss = torch.empty((), dtype=torch.float32, device=idx.device)
    grad = torch.empty((T, plan.k_tot), dtype=torch.float32, device=idx.device) if with_grad else None
    _check("dpb_variance_loss", load().dpb_variance_loss(
        plan._handle, _dev(idx, "idx"), _dev(coef, "coef"), T, int(n_min), _dev(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _dev(loss, "loss"), _opt(grad, "grad_coef"),
        _opt(grad_scale, "grad_scale"), _stream(idx)))
    return loss, grad


def variance_grad(plan: Plan, T: int, workspace: torch.Tensor, grad_scale: torch.Tensor | None = None,
                  grad: torch.Tensor | None = None):
    """Gradient of the variance loss from what a variance_loss call over T
    tokens left in `workspace`."""
    if grad is None:
        grad = torch.empty((T, plan.k_tot), dtype=torch.float32, device=workspace.device)
    _check("dpb_variance_grad", load().dpb_variance_grad(
        plan._handle, int(T), _dev(workspace, "workspace"), workspace.numel() * workspace.element_size(),
        _dev(grad, "grad_coef"), _opt(grad_scale, "grad_scale"), _stream(workspace)))
    return grad


STD_SAMPLE = 64


def std_state(plan: Plan, device=None):
    """Fresh standardization state (stats [N, 2] = (mu, r), m2 [N]) at its
    initial value (mu 0, r 1, m2 1)."""
    device = device or plan.device
    N = 1 << plan.level_bits[-1]
    stats = torch.empty((N, 2), dtype=torch.float32, device=device)
    m2 = torch.empty((N,), dtype=torch.float32, device=device)
    _check("dpb_std_init", load().dpb_std_init(plan._handle, _dev(stats, "stats"), _dev(m2, "m2"),
                                               _stream(stats)))
    return stats, m2


def encode_std(plan: Plan, x: torch.Tensor, stats: torch.Tensor, idx: torch.Tensor | None = None,
               coef: torch.Tensor | None = None, workspace: torch.Tensor | None = None):
    """Encoder on standardized scores z = (s - mu) r -> (idx, coef = z)."""
    assert stats.dtype == torch.float32 and stats.shape == (1 << plan.level_bits[-1], 2)
    return encode(plan, x, idx, coef, stats=stats, workspace=workspace)


def std_workspace(plan: Plan, device) -> torch.Tensor:
    n = int(load().dpb_std_workspace_bytes(plan._handle))
    return torch.empty(((n + 15) // 16) * 4, dtype=torch.float32, device=device)


def std_update(plan: Plan, x: torch.Tensor, idx: torch.Tensor, stats: torch.Tensor, m2: torch.Tensor,
               momentum: float, eps: float = 1e-6, workspace: torch.Tensor | None = None):
    """EMA update of (stats, m2) in place from the batch x and its code idx."""
    T = x.shape[0]
    assert idx.shape == (T, plan.k_tot) and idx.dtype == torch.int32
    if workspace is None:
        workspace = std_workspace(plan, x.device)
    _check("dpb_std_update", load().dpb_std_update(
        plan._handle, _dev(x, "x"), _dtype_code(x), T, _dev(idx, "idx"), float(momentum), float(eps),
        _dev(stats, "stats"), _dev(m2, "m2"), _dev(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _stream(x)))
    return stats, m2
