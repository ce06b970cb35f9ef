"""fp64 CPU oracle for PackMamba's packed causal conv1d and selective scan.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  It wraps the plain C
library built from ``oracle.c`` (no HIP, no shared code with the GPU path) and
takes numpy arrays; every floating input is converted to float64 exactly.

Functions and the passages they follow:
  conv1d_fwd / conv1d_bwd  -- Alg. 1 and §3.3 (taps stop at the sequence start)
  scan_fwd / scan_bwd      -- Eqs. (1a), (1b), (2a), Alg. 2 and §3.4
                              (A-bar forced to 0 where the position index is 0)
  scan_states              -- h at the end of every ``stride``-token chunk
  check_positions          -- the position-index contract of §3.1
Each operator optionally takes and returns per-row states for a sequence cut at
a row end and continued in another row (the future work of §5): the conv's width-1
inputs before the row / the row's last width-1 inputs, the scan's h before the
row / after it, with their gradients.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# PACKMAMBA_ORACLE_LIB names another build of oracle.c (e.g. a sanitizer build)
LIB_PATH = os.environ.get("PACKMAMBA_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
SRC_PATH = os.path.join(_HERE, "oracle.c")

_lib = None


def build(src: str = SRC_PATH, out: str = LIB_PATH, extra=()) -> str:
    """Compile the oracle with gcc (OpenMP, -O2, no fast-math) into ``out``."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-fno-fast-math",
           "-ffp-contract=off", "-I", _HERE, *extra, src, "-o", out, "-lm"]
    subprocess.run(cmd, check=True)
    return out


def load(path: Optional[str] = None):
    """Load (building first if absent) the oracle library; returns the ctypes handle."""
    global _lib
    if path is None and _lib is not None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        build(out=p)
    lib = ctypes.CDLL(p)
    dp, ip, i64, i32 = ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    lib.pmo_conv1d_fwd.argtypes = [dp, dp, dp, ip, dp, dp, dp, i64, i64, i64, i32, i32]
    lib.pmo_conv1d_bwd.argtypes = [dp, dp, dp, ip] + [dp] * 7 + [i64, i64, i64, i32, i32]
    lib.pmo_scan_fwd.argtypes = [dp] * 8 + [i32, ip, dp, dp, dp, i64, i64, i64, i32]
    lib.pmo_scan_states.argtypes = [dp, dp, dp, dp, dp, i32, ip, dp, dp, i64, i64, i64, i32, i64]
    lib.pmo_scan_bwd.argtypes = [dp] * 8 + [i32, ip] + [dp] * 12 + [i64, i64, i64, i32]
    lib.pmo_check_positions.argtypes = [ip, i64, i64, i32]
    lib.pmo_check_positions.restype = i64
    lib.pmo_num_threads.restype = i32
    lib.pmo_set_num_threads.argtypes = [i32]
    lib.pmo_set_num_threads.restype = None
    for f in (lib.pmo_conv1d_fwd, lib.pmo_conv1d_bwd, lib.pmo_scan_fwd, lib.pmo_scan_states,
              lib.pmo_scan_bwd):
        f.restype = None
    if path is None:
        _lib = lib
    return lib


def _f64(a):
    if a is None:
        return None
    return np.ascontiguousarray(a, dtype=np.float64)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _ptr(a):
    return None if a is None else a.ctypes.data


def num_threads(lib=None) -> int:
    return int((lib or load()).pmo_num_threads())


def set_num_threads(n: int, lib=None) -> None:
    (lib or load()).pmo_set_num_threads(int(n))


def conv1d_fwd(x, w, bias, pos, silu=True, lib=None, xinit=None, return_final=False):
    """out, or (out, xfinal) with ``return_final``; xinit/xfinal are (batch, dim, width-1)."""
    lib = lib or load()
    x, w, bias, pos, xinit = _f64(x), _f64(w), _f64(bias), _i32(pos), _f64(xinit)
    Nb, Dn, L = x.shape
    W = w.shape[1]
    out = np.empty_like(x)
    xfinal = np.empty((Nb, Dn, W - 1)) if return_final else None
    lib.pmo_conv1d_fwd(_ptr(x), _ptr(w), _ptr(bias), _ptr(pos), _ptr(xinit), _ptr(out), _ptr(xfinal),
                       Nb, Dn, L, W, int(silu))
    return (out, xfinal) if return_final else out


def conv1d_bwd(x, w, bias, pos, dout, silu=True, lib=None, xinit=None, dxfinal=None) -> Dict[str, np.ndarray]:
    lib = lib or load()
    x, w, bias, pos, dout = _f64(x), _f64(w), _f64(bias), _i32(pos), _f64(dout)
    xinit, dxfinal = _f64(xinit), _f64(dxfinal)
    Nb, Dn, L = x.shape
    W = w.shape[1]
    dx = np.empty_like(x)
    dw = np.empty_like(w)
    dbias = np.empty(Dn) if bias is not None else None
    dxinit = np.empty((Nb, Dn, W - 1)) if xinit is not None else None
    lib.pmo_conv1d_bwd(_ptr(x), _ptr(w), _ptr(bias), _ptr(pos), _ptr(xinit), _ptr(dout), _ptr(dxfinal),
                       _ptr(dx), _ptr(dw), _ptr(dbias), _ptr(dxinit), Nb, Dn, L, W, int(silu))
    return {"dx": dx, "dw": dw, "dbias": dbias, "dxinit": dxinit}


def scan_fwd(u, delta, A, B, C, D=None, z=None, delta_bias=None, delta_softplus=True, pos=None,
             lib=None, h0=None, return_final=False):
    """out, or (out, hfinal) with ``return_final``; h0/hfinal are (batch, dim, dstate)."""
    lib = lib or load()
    u, delta, A, B, C, D, z, delta_bias, h0 = map(_f64, (u, delta, A, B, C, D, z, delta_bias, h0))
    pos = _i32(pos)
    Nb, Dn, L = u.shape
    N = A.shape[1]
    out = np.empty_like(u)
    hfinal = np.empty((Nb, Dn, N)) if return_final else None
    lib.pmo_scan_fwd(_ptr(u), _ptr(delta), _ptr(A), _ptr(B), _ptr(C), _ptr(D), _ptr(z),
                     _ptr(delta_bias), int(delta_softplus), _ptr(pos), _ptr(h0), _ptr(out), _ptr(hfinal),
                     Nb, Dn, L, N)
    return (out, hfinal) if return_final else out


def scan_states(u, delta, A, B, delta_bias=None, delta_softplus=True, pos=None, stride=128,
                lib=None, h0=None) -> np.ndarray:
    lib = lib or load()
    u, delta, A, B, delta_bias, h0 = map(_f64, (u, delta, A, B, delta_bias, h0))
    pos = _i32(pos)
    Nb, Dn, L = u.shape
    N = A.shape[1]
    nchunk = (L + stride - 1) // stride
    st = np.empty((Nb, Dn, nchunk, N))
    lib.pmo_scan_states(_ptr(u), _ptr(delta), _ptr(A), _ptr(B), _ptr(delta_bias),
                        int(delta_softplus), _ptr(pos), _ptr(h0), _ptr(st), Nb, Dn, L, N, stride)
    return st


def scan_bwd(u, delta, A, B, C, D=None, z=None, delta_bias=None, delta_softplus=True, pos=None,
             dout=None, lib=None, h0=None, dhfinal=None) -> Dict[str, np.ndarray]:
    lib = lib or load()
    u, delta, A, B, C, D, z, delta_bias, dout = map(_f64, (u, delta, A, B, C, D, z, delta_bias, dout))
    h0, dhfinal = _f64(h0), _f64(dhfinal)
    pos = _i32(pos)
    Nb, Dn, L = u.shape
    N = A.shape[1]
    g = {
        "du": np.empty_like(u), "ddelta": np.empty_like(u), "dA": np.empty_like(A),
        "dB": np.empty_like(B), "dC": np.empty_like(C),
        "dD": np.empty(Dn) if D is not None else None,
        "dz": np.empty_like(u) if z is not None else None,
        "ddelta_bias": np.empty(Dn) if delta_bias is not None else None,
        "dh0": np.empty((Nb, Dn, N)) if h0 is not None else None,
    }
    lib.pmo_scan_bwd(_ptr(u), _ptr(delta), _ptr(A), _ptr(B), _ptr(C), _ptr(D), _ptr(z),
                     _ptr(delta_bias), int(delta_softplus), _ptr(pos), _ptr(h0), _ptr(dout), _ptr(dhfinal),
                     _ptr(g["du"]), _ptr(g["ddelta"]), _ptr(g["dA"]), _ptr(g["dB"]), _ptr(g["dC"]),
                     _ptr(g["dD"]), _ptr(g["dz"]), _ptr(g["ddelta_bias"]), _ptr(g["dh0"]), Nb, Dn, L, N)
    return g


def check_positions(pos, lib=None, continued=False) -> int:
    lib = lib or load()
    pos = _i32(pos)
    return int(lib.pmo_check_positions(_ptr(pos), pos.shape[0], pos.shape[1], int(continued)))
