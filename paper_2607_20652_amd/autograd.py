"""The DPB as a differentiable layer, and an MLP block that uses it.

`DPBLayer.apply(x, plan, normalized, n_min, std)` returns (y, loss_var):
  * forward: encode (§2.2 beam search; on standardized scores when a
    Standardizer is given), decode (§2.1), and, when `normalized`,
    the rescaling of the decoder output to ||x|| (§2.2 "Normalized
    Reconstruction"); loss_var is the variance auxiliary loss of the code
    (§2.2 "Auxillary losses"), or 0 when n_min is None; its per-slot
    pre-gradients stay in a workspace for the backward;
  * backward: the indices are held fixed and coef = Phi_S x (standardized:
    coef = (Phi_S x - mu) r), so
        grad_u    = backward of the normalization (dpb_normalize_bwd),
        grad_coef = Phi_S^T grad_u + g_loss * dL_var/dcoef,
        grad_x    = Phi_S (r grad_coef) + (the norm path of the normalization),
    all in the library's kernels: the normalization backward writes the
    norm-path term into the grad_x buffer and one dpb_decode_bwd_ex call adds
    the decode of grad_coef to it; a training backward then applies the EMA
    update of the standardization statistics from the batch.

`DPBMLP` places the layer in front of a GELU MLP with a residual connection
and RMSNorm, the position the paper's ParityTransformer gives it (§3.1: a
bottleneck before the input to every MLP).  The MLP's matrices are ordinary
torch layers; everything of the DPB itself runs in libdpb.so.
"""
from __future__ import annotations

import torch

from . import binding as B


class Standardizer:
    """EMA score-standardization state of one bottleneck (§2.2 "Score
    Standardization"): stats [N, 2] = (mu, r = 1/sigma) and m2 [N] (moving
    second raw moment), updated after every training backward with `momentum`."""

    def __init__(self, plan: B.Plan, momentum: float = 0.01, eps: float = 1e-6, device=None):
        self.plan, self.momentum, self.eps = plan, momentum, eps
        self.stats, self.m2 = B.std_state(plan, device)
        self.workspace = B.std_workspace(plan, self.stats.device)
        self.training = True

    def update(self, x: torch.Tensor, idx: torch.Tensor):
        B.std_update(self.plan, x, idx, self.stats, self.m2, self.momentum, self.eps, self.workspace)


class DPBLayer(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x: torch.Tensor, plan: B.Plan, normalized: bool = True, n_min: int | None = None,
                std: Standardizer | None = None):
        x = x.contiguous()
        idx, coef = B.encode_std(plan, x, std.stats) if std is not None else B.encode(plan, x)
        u = B.decode(plan, idx, coef, x.dtype)
        y = B.normalize(plan, u, x) if normalized else u
        ws = None
        if n_min is not None:
            ws = B.variance_workspace(plan, x.shape[0], x.device)
            loss, _ = B.variance_loss(plan, idx, coef, n_min, with_grad=False, workspace=ws)
        else:
            loss = torch.zeros((), dtype=torch.float32, device=x.device)
        ctx.plan, ctx.normalized, ctx.n_min, ctx.std = plan, normalized, n_min, std
        ctx.save_for_backward(x, idx, coef, u, ws)
        ctx.set_materialize_grads(False)
        return y, loss

    @staticmethod
    def backward(ctx, gy: torch.Tensor | None, gloss: torch.Tensor | None):
        plan = ctx.plan
        x, idx, coef, u, ws = ctx.saved_tensors
        if gy is None:
            gy = torch.zeros_like(x)
        gy = gy.contiguous()
        if ctx.normalized:
            gu, gx = B.normalize_bwd(plan, gy, u, x, gu_dtype=gy.dtype, gr_dtype=x.dtype)
        else:
            gu, gx = gy, None
        add_gc = None
        if gloss is not None and ctx.n_min is not None:
            # the forward left the per-slot pre-gradients in ws
            add_gc = B.variance_grad(plan, x.shape[0], ws, grad_scale=gloss.to(torch.float32).contiguous())
        std = ctx.std
        _, gx = B.decode_bwd_ex(plan, idx, gu, add_grad_coef=add_gc, add_grad_x=gx, gx_dtype=x.dtype, grad_x=gx,
                                stats=std.stats if std is not None else None)
        if std is not None and std.training:
            # the statistics this batch was encoded with are no longer needed
            std.update(x, idx)
        return gx, None, None, None, None


def dpb_layer(x: torch.Tensor, plan: B.Plan, normalized: bool = True, n_min: int | None = None,
              std: Standardizer | None = None):
    """Functional form of DPBLayer: (y, loss_var)."""
    return DPBLayer.apply(x, plan, normalized, n_min, std)


class DPBMLP(torch.nn.Module):
    """h + W2 gelu(W1 DPB(rmsnorm(h))): a transformer MLP sublayer with the
    parity bottleneck at its input.  forward returns (output, loss_var)."""

    def __init__(self, plan: B.Plan, d_ff: int, normalized: bool = True, n_min: int | None = None,
                 standardize: bool = False, momentum: float = 0.01, dtype: torch.dtype = torch.float32, device=None):
        super().__init__()
        d = plan.d
        self.plan, self.normalized, self.n_min = plan, normalized, n_min
        self.std = Standardizer(plan, momentum, device=device) if standardize else None
        if self.std is not None:
            self.register_buffer("std_stats", self.std.stats)
            self.register_buffer("std_m2", self.std.m2)
        self.norm = torch.nn.RMSNorm(d, dtype=dtype, device=device)
        self.fc1 = torch.nn.Linear(d, d_ff, dtype=dtype, device=device)
        self.fc2 = torch.nn.Linear(d_ff, d, dtype=dtype, device=device)

    def forward(self, h: torch.Tensor):
        shape = h.shape
        z = self.norm(h).reshape(-1, shape[-1])
        if self.std is not None:
            self.std.training = self.training
        y, loss_var = DPBLayer.apply(z, self.plan, self.normalized, self.n_min, self.std)
        out = h + self.fc2(torch.nn.functional.gelu(self.fc1(y))).reshape(shape)
        return out, loss_var
