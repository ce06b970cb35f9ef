"""A packed Mamba-1 block on one GPU (§3.2): RMSNorm, input projection, packed causal
conv1d + SiLU, x and dt projections, packed selective scan with the D skip and the
SiLU(z) gate, output projection, residual -- forward and backward.

The sequence-wise steps (conv, scan) and RMSNorm (with the residual's gradient
folded into its backward) run in this library's HIP kernels through the C ABI; the
projections are plain GEMMs, run by hipBLASLt through torch.matmul / baddbmm, which
also add the residual and accumulate the two-term input gradients (§3.2: token-wise and
element-wise operators satisfy PUI unchanged, so packing needs nothing from them).  Activations are
laid out (batch, features, seqlen), sequence innermost, which is the layout of the
conv and scan kernels, so no transposes sit between the steps: each projection is a
batched GEMM W @ X[b], split per output part so that every tensor the kernels see is
contiguous.

Parameters (dict of tensors on the device): norm_w (d_model), W_in (2*d_inner,
d_model), conv_w (d_inner, W), conv_b (d_inner), W_x (R + 2N, d_inner), W_dt (d_inner,
R), dt_bias (d_inner), A (d_inner, N), D (d_inner), W_out (d_model, d_inner).  The
projection weights are in the activation dtype; the others are fp32.
"""
from __future__ import annotations

from typing import Callable, Dict, Optional

import paper_2408_03865_amd as P

EPS = 1e-5


def _torch():
    import torch
    return torch


def _lin(W, X):
    """Y[b] = W @ X[b]; X (batch, in, L) contiguous."""
    return _torch().matmul(W, X)


def _lin_dx(W, dY):
    """dX[b] = W^T @ dY[b]."""
    return _torch().matmul(W.t().contiguous(), dY)


def _lin_dw(dY, X):
    """dW = sum_b dY[b] @ X[b]^T: one 2-D GEMM per batch row, X[b] read transposed in
    place (no copy), accumulated in fp32 in place (a new accumulator per row would be
    copied first) and returned in dY's dtype."""
    torch = _torch()
    f32 = torch.float32
    kw = {} if dY.dtype == f32 else {"out_dtype": f32}
    acc = torch.mm(dY[0], X[0].t(), **kw)
    for b in range(1, dY.shape[0]):
        torch.addmm(acc, dY[b], X[b].t(), out=acc, **kw)
    return acc.to(dY.dtype)


def _lin_dw_thin(dY, X):
    """dW = sum_b dY[b] @ X[b]^T for a thin weight (one side of at most a few hundred
    rows): one batched GEMM with fp32 outputs, summed over the batch (2.3x faster than
    the per-row chain for the x and dt projections).  The thin operand is the one
    copied transposed: right operands of batched bf16 products are kept contiguous."""
    torch = _torch()
    kw = {} if dY.dtype == torch.float32 else {"out_dtype": torch.float32}
    if dY.shape[1] <= X.shape[1]:
        acc = torch.bmm(X, dY.transpose(1, 2).contiguous(), **kw).sum(0).t()
    else:
        acc = torch.bmm(dY, X.transpose(1, 2).contiguous(), **kw).sum(0)
    return acc.to(dY.dtype).contiguous()


def _bcast(W, batch):
    """W as the batched left operand of a GEMM (stride 0 over the batch)."""
    return W.contiguous().expand(batch, -1, -1)


def block_forward(x, pos, p: Dict[str, object], mark: Optional[Callable[[str], None]] = None):
    """out = x + W_out @ scan(conv(W_in,x @ RMSNorm(x)), ...): returns (out, ctx)."""
    mk = mark or (lambda name: None)
    Dn = p["D"].shape[0]
    N = p["A"].shape[1]
    R = p["W_dt"].shape[1]
    mk("norm")
    h, r = P.rmsnorm_fwd(x, p["norm_w"], EPS)
    mk("in_proj")
    xi = _lin(p["W_in"][:Dn], h)
    z = _lin(p["W_in"][Dn:], h)
    mk("conv")
    u = P.causal_conv1d_fwd(xi, p["conv_w"], p["conv_b"], pos, silu=True)
    mk("x_proj")
    Wx = p["W_x"]
    dtl = _lin(Wx[:R], u)
    B = _lin(Wx[R:R + N], u)
    C = _lin(Wx[R + N:], u)
    delta = _lin(p["W_dt"], dtl)
    mk("scan")
    y, st = P.selective_scan_fwd(u, delta, p["A"], B, C, p["D"], z, p["dt_bias"], True, pos,
                                 return_states=True)
    mk("out_proj")
    out = _torch().baddbmm(x, _bcast(p["W_out"], x.shape[0]), y)    # the residual added by the GEMM
    mk("end")
    ctx = dict(x=x, pos=pos, h=h, r=r, xi=xi, z=z, u=u, dtl=dtl, B=B, C=C, delta=delta, y=y, st=st)
    return out, ctx


def block_backward(dout, ctx, p, mark: Optional[Callable[[str], None]] = None,
                   trace: Optional[Dict[str, object]] = None) -> Dict[str, object]:
    """Gradients of sum(dout * out) with respect to x and every parameter.  With ``trace``
    (a dict), the backward's own intermediates are left in it: the scan's upstream
    gradient dy and its outputs scan (scan_du: its du before the x projection's
    gradient is added in place), the conv's upstream gradient du and its dx dxi,
    and the RMSNorm's upstream gradient dh."""
    mk = mark or (lambda name: None)
    Dn = p["D"].shape[0]
    Wx = p["W_x"]
    dt = dout.dtype
    g = {}
    mk("out_proj_bwd")
    g["W_out"] = _lin_dw(dout, ctx["y"])
    dy = _lin_dx(p["W_out"], dout)
    mk("scan_bwd")
    s = P.selective_scan_bwd(ctx["u"], ctx["delta"], p["A"], ctx["B"], ctx["C"], p["D"], ctx["z"],
                             p["dt_bias"], True, ctx["pos"], dy, saved_states=ctx["st"])
    g["A"], g["D"], g["dt_bias"] = s["dA"], s["dD"], s["ddelta_bias"]
    mk("x_proj_bwd")
    g["W_dt"] = _lin_dw_thin(s["ddelta"], ctx["dtl"])
    ddtl = _lin_dx(p["W_dt"], s["ddelta"])
    dxdbl = _torch().cat([ddtl, s["dB"].to(dt), s["dC"].to(dt)], 1)      # (batch, R + 2N, L)
    g["W_x"] = _lin_dw_thin(dxdbl, ctx["u"])
    if trace is not None:
        trace["scan_du"] = s["du"].clone()       # the scan's own du, before the sum below
    du = s["du"].baddbmm_(_bcast(Wx.t(), dxdbl.shape[0]), dxdbl)   # accumulated into the scan's du
    mk("conv_bwd")
    dxi, g["conv_w"], g["conv_b"] = P.causal_conv1d_bwd(ctx["xi"], p["conv_w"], p["conv_b"], ctx["pos"],
                                                        du.contiguous(), silu=True)
    mk("in_proj_bwd")
    g["W_in"] = _torch().cat([_lin_dw(dxi, ctx["h"]), _lin_dw(s["dz"], ctx["h"])], 0)
    dh = _lin_dx(p["W_in"][:Dn], dxi)
    dh.baddbmm_(_bcast(p["W_in"][Dn:].t(), dh.shape[0]), s["dz"])
    mk("norm_bwd")
    # the residual's gradient (dout itself) is added inside the RMSNorm backward
    g["x"], g["norm_w"] = P.rmsnorm_bwd(ctx["x"], p["norm_w"], ctx["r"], dh, dresidual=dout)
    mk("end")
    if trace is not None:
        trace.update(dy=dy, scan=s, du=du, dxi=dxi, dh=dh)
    return g
