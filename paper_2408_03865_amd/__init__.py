"""PackMamba's packed causal conv1d and selective scan on MI355X (gfx950).

Thin torch-facing wrappers over the C ABI of ``libpackmamba.so`` (see
``include/packmamba.h``).  They allocate outputs and workspace with torch on
the tensors' device, pass raw pointers and the current stream, and check the
status.  Nothing is computed here.

    out = causal_conv1d_fwd(x, weight, bias, position_indices, silu=True)
    dx, dweight, dbias = causal_conv1d_bwd(x, weight, bias, position_indices, dout, silu=True)
    out, states = selective_scan_fwd(u, delta, A, B, C, D, z, delta_bias, True, position_indices,
                                     return_states=True)
    grads = selective_scan_bwd(u, delta, A, B, C, D, z, delta_bias, True, position_indices, dout,
                               saved_states=states)

A sequence cut at a row end continues in another row when the second part is given
the first part's final states (the future work of §5):
    out1, xf = causal_conv1d_fwd(x1, w, bias, pos1, return_final=True)
    out2 = causal_conv1d_fwd(x2, w, bias, pos2, initial_x=xf)
    y1, hf = selective_scan_fwd(..., pos1, return_final=True)
    y2 = selective_scan_fwd(..., pos2, initial_state=hf)
and in the backward the second part's initial-state gradients are the first part's
final-state gradients (dfinal_x, dfinal_state).
"""
from __future__ import annotations

from typing import Dict, Optional

from . import _lib
from ._lib import BF16, BF16_F32OUT, F32, STATE_STRIDE, PackMambaError, load

__all__ = [
    "causal_conv1d_fwd", "causal_conv1d_bwd", "selective_scan_fwd", "selective_scan_bwd",
    "check_position_indices", "saved_states_size", "chunk_states", "segments", "pack_plan",
    "pack_positions",
    "rmsnorm_fwd", "rmsnorm_bwd",
    "padding_rate", "PackMambaError", "load", "F32", "BF16",
    "STATE_STRIDE", "BF16_F32OUT",
]


def _torch():
    import torch
    return torch


def _code(t, out_f32: bool = False) -> int:
    torch = _torch()
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16_F32OUT if out_f32 else BF16
    raise TypeError(f"unsupported activation dtype {t.dtype}")


def _empty_out(t, out_f32: bool):
    torch = _torch()
    return torch.empty(t.shape, dtype=torch.float32 if out_f32 else t.dtype, device=t.device)


def _p(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(t) -> int:
    return _torch().cuda.current_stream(t.device).cuda_stream


def _workspace(nbytes: int, device):
    torch = _torch()
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def causal_conv1d_fwd(x, weight, bias, position_indices, silu: bool = True, out_f32: bool = False,
                      initial_x=None, return_final: bool = False):
    """out_f32: for bf16 x, return fp32 outputs (the values before the bf16 rounding).
    initial_x: (batch, dim, width-1) in x's dtype; return_final adds the row's last
    width-1 inputs to the result."""
    torch = _torch()
    Nb, Dn, L = x.shape
    W = weight.shape[1]
    out = _empty_out(x, out_f32)
    fin = torch.empty((Nb, Dn, W - 1), dtype=x.dtype, device=x.device) if return_final else None
    st = load().packmamba_causal_conv1d_fwd(_p(x), _p(weight), _p(bias), _p(position_indices),
                                            _p(initial_x), _p(out), _p(fin), Nb, Dn, L, W,
                                            _code(x, out_f32), int(silu), _stream(x))
    _lib.check("packmamba_causal_conv1d_fwd", st)
    return (out, fin) if return_final else out


def causal_conv1d_bwd(x, weight, bias, position_indices, dout, silu: bool = True, workspace=None,
                      out_f32: bool = False, initial_x=None, dfinal_x=None):
    """(dx, dweight, dbias), plus dinitial_x when initial_x is given."""
    torch = _torch()
    Nb, Dn, L = x.shape
    W = weight.shape[1]
    lib = load()
    dx = _empty_out(x, out_f32)
    dw = torch.empty_like(weight)
    db = torch.empty_like(bias) if bias is not None else None
    dinit = None
    if initial_x is not None:
        dinit = torch.empty((Nb, Dn, W - 1), dtype=dx.dtype, device=x.device)
    need = lib.packmamba_causal_conv1d_bwd_workspace_size(Nb, Dn, L, W)
    ws = workspace if workspace is not None else _workspace(need, x.device)
    st = lib.packmamba_causal_conv1d_bwd(_p(x), _p(weight), _p(bias), _p(position_indices), _p(initial_x),
                                         _p(dout), _p(dfinal_x), _p(dx), _p(dw), _p(db), _p(dinit),
                                         _p(ws), ws.numel(), Nb, Dn, L, W, _code(x, out_f32), int(silu),
                                         _stream(x))
    _lib.check("packmamba_causal_conv1d_bwd", st)
    return (dx, dw, db) if initial_x is None else (dx, dw, db, dinit)


def rmsnorm_fwd(x, weight, eps: float = 1e-5, out_f32: bool = False):
    """RMSNorm over the feature axis of x (batch, dim, seqlen): (out, rstd), rstd
    (batch, seqlen) fp32 for the backward."""
    torch = _torch()
    Nb, Dn, L = x.shape
    out = _empty_out(x, out_f32)
    rstd = torch.empty((Nb, L), dtype=torch.float32, device=x.device)
    st = load().packmamba_rmsnorm_fwd(_p(x), _p(weight), float(eps), _p(out), _p(rstd), Nb, Dn, L,
                                      _code(x, out_f32), _stream(x))
    _lib.check("packmamba_rmsnorm_fwd", st)
    return out, rstd


def rmsnorm_bwd(x, weight, rstd, dout, dresidual=None, workspace=None, out_f32: bool = False):
    """(dx, dweight); dresidual, if given, is added to dx (a residual connection)."""
    torch = _torch()
    Nb, Dn, L = x.shape
    lib = load()
    dx = _empty_out(x, out_f32)
    dw = torch.empty_like(weight)
    need = lib.packmamba_rmsnorm_bwd_workspace_size(Nb, Dn, L)
    ws = workspace if workspace is not None else _workspace(need, x.device)
    st = lib.packmamba_rmsnorm_bwd(_p(x), _p(weight), _p(rstd), _p(dout), _p(dresidual), _p(dx), _p(dw),
                                   _p(ws), ws.numel(), Nb, Dn, L, _code(x, out_f32), _stream(x))
    _lib.check("packmamba_rmsnorm_bwd", st)
    return dx, dw


def segments(batch: int, dim: int, seqlen: int, direction: str = "bwd") -> int:
    """Segments per row the scan forward ("fwd") or backward ("bwd") uses for this shape
    (1: rows are not split).  Mirrors the rule of the library's launchers, for tests and
    reports only."""
    target = {"fwd": 768, "bwd": 1536}[direction]
    blocks = batch * ((dim + 15) // 16)
    units = (seqlen + 255) // 256
    if blocks * 2 >= target or units < 2:
        return 1
    nseg = min((target + blocks - 1) // blocks, units)
    per = (units + nseg - 1) // nseg
    return (units + per - 1) // per


def saved_states_size(batch: int, dim: int, seqlen: int, dstate: int = 16) -> int:
    return int(load().packmamba_selective_scan_fwd_saved_states_size(batch, dim, seqlen, dstate))


def chunk_states(saved_states, batch: int, dim: int, seqlen: int, dstate: int = 16):
    """The chunk states inside a saved-states buffer: (batch, dim, chunk, dstate), h after
    token min((c+1) STATE_STRIDE, seqlen) - 1 of chunk c."""
    nch = (seqlen + STATE_STRIDE - 1) // STATE_STRIDE
    return saved_states[:batch * dim * nch * dstate].view(batch, dim, nch, dstate)


def selective_scan_fwd(u, delta, A, B, C, D, z, delta_bias, delta_softplus, position_indices,
                       return_states: bool = False, out=True, out_f32: bool = False, workspace=None,
                       initial_state=None, return_final: bool = False):
    """out, followed by the saved states (return_states: a flat fp32 buffer for the
    backward, holding the chunk states, see chunk_states, and the dz factor) and the
    final state (return_final, (batch, dim, dstate) fp32) when asked for; initial_state
    is (batch, dim, dstate) fp32."""
    torch = _torch()
    Nb, Dn, L = u.shape
    N = A.shape[1]
    lib = load()
    o = _empty_out(u, out_f32) if out else None
    need = int(lib.packmamba_selective_scan_fwd_workspace_size(Nb, Dn, L, N))
    ws = workspace if workspace is not None or need == 0 else _workspace(need, u.device)
    states = None
    if return_states:
        nbytes = int(lib.packmamba_selective_scan_fwd_saved_states_size(Nb, Dn, L, N))
        states = torch.empty(nbytes // 4, dtype=torch.float32, device=u.device)
    fin = torch.empty((Nb, Dn, N), dtype=torch.float32, device=u.device) if return_final else None
    st = lib.packmamba_selective_scan_fwd(
        _p(u), _p(delta), _p(A), _p(B), _p(C), _p(D), _p(z), _p(delta_bias), int(delta_softplus),
        _p(position_indices), _p(initial_state), _p(o), _p(fin), _p(states), _p(ws),
        0 if ws is None else ws.numel(), Nb, Dn, L, N, _code(u, out_f32), _stream(u))
    _lib.check("packmamba_selective_scan_fwd", st)
    res = (o,) + ((states,) if return_states else ()) + ((fin,) if return_final else ())
    return res if len(res) > 1 else o


def selective_scan_bwd(u, delta, A, B, C, D, z, delta_bias, delta_softplus, position_indices, dout,
                       saved_states=None, workspace=None, out_f32: bool = False, initial_state=None,
                       dfinal_state=None) -> Dict[str, object]:
    torch = _torch()
    Nb, Dn, L = u.shape
    N = A.shape[1]
    lib = load()
    g = {
        "du": _empty_out(u, out_f32), "ddelta": _empty_out(u, out_f32), "dA": torch.empty_like(A),
        "dB": torch.empty(B.shape, dtype=torch.float32, device=u.device),
        "dC": torch.empty(C.shape, dtype=torch.float32, device=u.device),
        "dD": torch.empty_like(D) if D is not None else None,
        "dz": _empty_out(z, out_f32) if z is not None else None,
        "ddelta_bias": torch.empty_like(delta_bias) if delta_bias is not None else None,
        "dinitial_state": torch.empty_like(initial_state) if initial_state is not None else None,
    }
    need = lib.packmamba_selective_scan_bwd_workspace_size(Nb, Dn, L, N)
    ws = workspace if workspace is not None else _workspace(need, u.device)
    st = lib.packmamba_selective_scan_bwd(
        _p(u), _p(delta), _p(A), _p(B), _p(C), _p(D), _p(z), _p(delta_bias), int(delta_softplus),
        _p(position_indices), _p(initial_state), _p(dout), _p(dfinal_state), _p(saved_states),
        _p(g["du"]), _p(g["ddelta"]), _p(g["dA"]), _p(g["dB"]), _p(g["dC"]), _p(g["dD"]), _p(g["dz"]),
        _p(g["ddelta_bias"]), _p(g["dinitial_state"]), _p(ws), ws.numel(),
        Nb, Dn, L, N, _code(u, out_f32), _stream(u))
    _lib.check("packmamba_selective_scan_bwd", st)
    return g


def check_position_indices(position_indices, continued: bool = False) -> bool:
    """True if the indices satisfy the packing contract (checked on the device);
    with ``continued``, rows may start inside a sequence carried over from another row."""
    torch = _torch()
    flag = torch.zeros(4, dtype=torch.int32, device=position_indices.device)
    Nb, L = position_indices.shape
    st = load().packmamba_check_position_indices(_p(position_indices), Nb, L, int(continued), _p(flag),
                                                 _stream(position_indices))
    _lib.check("packmamba_check_position_indices", st)
    return int(flag[0].item()) == 0


_POLICIES = {"sequential": _lib.PACK_SEQUENTIAL, "greedy": _lib.PACK_GREEDY, "cut": _lib.PACK_CUT}


def pack_plan(lengths, seqlen: int, policy: str = "sequential", window: int = 64):
    """Host packing plan of a stream of sequence lengths (the library's C++ planner):
    returns (pieces, n_rows), pieces an int64 array (n, 5) of (seq, row, offset,
    length, first_pos).  Policies: "sequential" (seal a row when the next sequence
    does not fit), "greedy" (windows of ``window`` sequences sorted longest first,
    first-fit), "cut" (rows filled to the end, sequences cut and continued in the
    next row; needs the operators' state passing)."""
    import ctypes
    import numpy as np
    lib = load()
    ln = np.ascontiguousarray(lengths, dtype=np.int64)
    n_pieces, n_rows = ctypes.c_int64(), ctypes.c_int64()
    pol = _POLICIES[policy]
    _lib.check("packmamba_pack_plan", lib.packmamba_pack_plan(
        ln.ctypes.data, ln.size, seqlen, pol, window, None, 0, ctypes.byref(n_pieces), ctypes.byref(n_rows)))
    out = np.zeros((n_pieces.value, 5), dtype=np.int64)
    _lib.check("packmamba_pack_plan", lib.packmamba_pack_plan(
        ln.ctypes.data, ln.size, seqlen, pol, window, out.ctypes.data, n_pieces.value,
        ctypes.byref(n_pieces), ctypes.byref(n_rows)))
    return out, int(n_rows.value)


def pack_positions(pieces, n_rows: int, seqlen: int):
    """Host int32 position indices (n_rows, seqlen) of a plan (padding tokens get 0)."""
    import numpy as np
    pc = np.ascontiguousarray(pieces, dtype=np.int64)
    pos = np.empty((n_rows, seqlen), dtype=np.int32)
    _lib.check("packmamba_pack_positions", load().packmamba_pack_positions(
        pc.ctypes.data if pc.size else None, pc.shape[0], n_rows, seqlen, pos.ctypes.data))
    return pos


def padding_rate(pieces, n_rows: int, seqlen: int) -> float:
    """Fraction of the rows' tokens that hold no sequence."""
    import numpy as np
    return 1.0 - float(np.asarray(pieces)[:, 3].sum()) / float(max(1, n_rows * seqlen))
