"""fp64 CPU reference of one packed Mamba-1 block (§3.2): RMSNorm, the input
projection, the packed causal conv1d with SiLU, the x and dt projections, the packed
selective scan with its D skip and SiLU(z) gate, the output projection and the
residual.

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``.  It composes the oracle's
sequence-wise operators (Alg. 1, Alg. 2) with token-wise steps written out in numpy
(§3.2 classes (i) and (ii): RMSNorm and the linear layers, which satisfy PUI as
they are).  Layout: activations (batch, features, seqlen), sequence innermost.

Parameters (dict): norm_w (d_model), W_in (2*d_inner, d_model), conv_w (d_inner, W),
conv_b (d_inner), W_x (R + 2N, d_inner), W_dt (d_inner, R), dt_bias (d_inner),
A (d_inner, N), D (d_inner), W_out (d_model, d_inner).
"""
from __future__ import annotations

from typing import Dict

import numpy as np

from . import conv1d_bwd, conv1d_fwd, scan_bwd, scan_fwd

EPS = 1e-5


def _lin(W, X):
    """Y[b] = W @ X[b] for X (batch, in, L)."""
    return np.einsum("oi,bil->bol", W, X)


def _lin_grads(W, X, dY):
    """Gradients of Y = W @ X: (dW, dX)."""
    return np.einsum("bol,bil->oi", dY, X), np.einsum("oi,bol->bil", W, dY)


def rmsnorm(x, w, eps=EPS):
    """x * w / sqrt(mean_d x^2 + eps), over the feature axis (1) at each token."""
    r = 1.0 / np.sqrt(np.mean(x * x, axis=1, keepdims=True) + eps)
    return x * r * w[None, :, None], r


def rmsnorm_bwd(x, w, r, dh):
    xh = x * r
    dw = np.sum(dh * xh, axis=(0, 2))
    dxh = dh * w[None, :, None]
    dx = r * (dxh - xh * np.mean(dxh * xh, axis=1, keepdims=True))
    return dx, dw


def block_fwd(x, pos, p: Dict[str, np.ndarray], keep: bool = False):
    """Returns out (batch, d_model, L) = x + W_out @ scan(...); with keep, also the
    intermediates the backward uses."""
    Dn = p["D"].shape[0]
    N = p["A"].shape[1]
    R = p["W_dt"].shape[1]
    h, r = rmsnorm(x, p["norm_w"])
    xz = _lin(p["W_in"], h)
    xi, z = xz[:, :Dn], xz[:, Dn:]
    u = conv1d_fwd(xi, p["conv_w"], p["conv_b"], pos, silu=True)
    xdbl = _lin(p["W_x"], u)
    dtl, B, C = xdbl[:, :R], xdbl[:, R:R + N], xdbl[:, R + N:]
    delta = _lin(p["W_dt"], dtl)
    y = scan_fwd(u, delta, p["A"], B, C, p["D"], z, p["dt_bias"], True, pos)
    out = x + _lin(p["W_out"], y)
    if not keep:
        return out
    return out, dict(h=h, r=r, xi=xi, z=z, u=u, dtl=dtl, B=B, C=C, delta=delta, y=y)


def block_bwd(x, pos, p, dout) -> Dict[str, np.ndarray]:
    """Gradients of sum(dout * block_fwd(x)) with respect to x and every parameter."""
    Dn = p["D"].shape[0]
    _, c = block_fwd(x, pos, p, keep=True)
    g = {}
    g["W_out"], dy = _lin_grads(p["W_out"], c["y"], dout)
    s = scan_bwd(c["u"], c["delta"], p["A"], c["B"], c["C"], p["D"], c["z"], p["dt_bias"], True, pos, dout=dy)
    g["A"], g["D"], g["dt_bias"] = s["dA"], s["dD"], s["ddelta_bias"]
    g["W_dt"], ddtl = _lin_grads(p["W_dt"], c["dtl"], s["ddelta"])
    dxdbl = np.concatenate([ddtl, s["dB"], s["dC"]], axis=1)
    g["W_x"], du2 = _lin_grads(p["W_x"], c["u"], dxdbl)
    cg = conv1d_bwd(c["xi"], p["conv_w"], p["conv_b"], pos, s["du"] + du2, silu=True)
    g["conv_w"], g["conv_b"] = cg["dw"], cg["dbias"]
    dxz = np.concatenate([cg["dx"], s["dz"]], axis=1)
    g["W_in"], dh = _lin_grads(p["W_in"], c["h"], dxz)
    dxn, g["norm_w"] = rmsnorm_bwd(x, p["norm_w"], c["r"], dh)
    g["x"] = dout + dxn
    return g
