"""The DPB as a differentiable layer, and an MLP block that uses it.

`DPBLayer.apply(x, plan, normalized, n_min)` returns (y, loss_var):
  * forward: encode (§2.2 beam search), decode (§2.1), and, when `normalized`,
    the rescaling of the decoder output to ||x|| (§2.2 "Normalized
    Reconstruction"); loss_var is the variance auxiliary loss of the code
    (§2.2 "Auxillary losses"), or 0 when n_min is None; its per-slot
    pre-gradients stay in a workspace for the backward;
  * backward: the indices are held fixed and coef = Phi_S x, so
        grad_u    = backward of the normalization (dpb_normalize_bwd),
        grad_coef = Phi_S^T grad_u + g_loss * dL_var/dcoef,
        grad_x    = Phi_S grad_coef + (the norm path of the normalization),
    all in the library's kernels: the normalization backward writes the
    norm-path term into the grad_x buffer and one dpb_decode_bwd_ex call adds
    the decode of grad_coef to it.

`DPBMLP` places the layer in front of a GELU MLP with a residual connection
and RMSNorm, the position the paper's ParityTransformer gives it (§3.1: a
bottleneck before the input to every MLP).  The MLP's matrices are ordinary
torch layers; everything of the DPB itself runs in libdpb.so.
"""
from __future__ import annotations

import torch

from . import binding as B


class DPBLayer(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x: torch.Tensor, plan: B.Plan, normalized: bool = True, n_min: int | None = None):
        x = x.contiguous()
        idx, coef = B.encode(plan, x)
        u = B.decode(plan, idx, coef, x.dtype)
        y = B.normalize(plan, u, x) if normalized else u
        ws = None
        if n_min is not None:
            ws = B.variance_workspace(plan, x.shape[0], x.device)
            loss, _ = B.variance_loss(plan, idx, coef, n_min, with_grad=False, workspace=ws)
        else:
            loss = torch.zeros((), dtype=torch.float32, device=x.device)
        ctx.plan, ctx.normalized, ctx.n_min = plan, normalized, n_min
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
        _, gx = B.decode_bwd_ex(plan, idx, gu, add_grad_coef=add_gc, add_grad_x=gx, gx_dtype=x.dtype, grad_x=gx)
        return gx, None, None, None


def dpb_layer(x: torch.Tensor, plan: B.Plan, normalized: bool = True, n_min: int | None = None):
    """Functional form of DPBLayer: (y, loss_var)."""
    return DPBLayer.apply(x, plan, normalized, n_min)


class DPBMLP(torch.nn.Module):
    """h + W2 gelu(W1 DPB(rmsnorm(h))): a transformer MLP sublayer with the
    parity bottleneck at its input.  forward returns (output, loss_var)."""

    def __init__(self, plan: B.Plan, d_ff: int, normalized: bool = True, n_min: int | None = None,
                 dtype: torch.dtype = torch.float32, device=None):
        super().__init__()
        d = plan.d
        self.plan, self.normalized, self.n_min = plan, normalized, n_min
        self.norm = torch.nn.RMSNorm(d, dtype=dtype, device=device)
        self.fc1 = torch.nn.Linear(d, d_ff, dtype=dtype, device=device)
        self.fc2 = torch.nn.Linear(d_ff, d, dtype=dtype, device=device)

    def forward(self, h: torch.Tensor):
        shape = h.shape
        z = self.norm(h).reshape(-1, shape[-1])
        y, loss_var = DPBLayer.apply(z, self.plan, self.normalized, self.n_min)
        out = h + self.fc2(torch.nn.functional.gelu(self.fc1(y))).reshape(shape)
        return out, loss_var
