"""ctypes binding of libpackmamba.so: the C ABI in include/packmamba.h, same names.

Argument marshalling only.  Every step of the path runs in the HIP kernels of
the library; torch provides device memory and the current stream.  There is no
fallback: if the library is missing or was not built for this GPU, loading
raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
# PACKMAMBA_LIB names another build of the library (e.g. a host-side sanitizer build)
LIB_PATH = os.environ.get("PACKMAMBA_LIB") or os.path.join(HERE, "libpackmamba.so")

F32, BF16, BF16_F32OUT = 0, 1, 2
STATE_STRIDE = 128
ABI_VERSION = 6

STATUS = {0: "OK", 1: "ERR_NULL", 2: "ERR_SHAPE", 3: "ERR_UNSUPPORTED", 4: "ERR_ALIGN",
          5: "ERR_WORKSPACE", 6: "ERR_LAUNCH", 7: "ERR_SCRATCH"}
NOALLOC_SCRATCH_BYTES = 16 << 20

# Every symbol the header declares.
EXPORTS = (
    "packmamba_abi_version", "packmamba_status_string",
    "packmamba_causal_conv1d_fwd", "packmamba_causal_conv1d_bwd_workspace_size",
    "packmamba_causal_conv1d_bwd", "packmamba_selective_scan_fwd_saved_states_size",
    "packmamba_selective_scan_fwd_workspace_size", "packmamba_selective_scan_fwd",
    "packmamba_selective_scan_bwd_workspace_size", "packmamba_selective_scan_bwd",
    "packmamba_check_position_indices", "packmamba_pack_plan", "packmamba_pack_positions",
    "packmamba_rmsnorm_fwd", "packmamba_rmsnorm_bwd_workspace_size", "packmamba_rmsnorm_bwd",
    "packmamba_causal_conv1d_bwd_noalloc",
)

PACK_SEQUENTIAL, PACK_GREEDY, PACK_CUT = 0, 1, 2


class Piece(ctypes.Structure):
    """packmamba_piece: one sequence's piece in a packing plan."""
    _fields_ = [("seq", ctypes.c_int64), ("row", ctypes.c_int64), ("offset", ctypes.c_int64),
                ("length", ctypes.c_int64), ("first_pos", ctypes.c_int64)]


class PackMambaError(RuntimeError):
    def __init__(self, fn: str, status: int, text: str):
        super().__init__(f"{fn}: {STATUS.get(status, status)} ({text})")
        self.status = status


_lib = None
_lib_path = None   # the file _lib was loaded from


def load(path: Optional[str] = None) -> ctypes.CDLL:
    """Load the HIP library (raises if it is absent: build with paper_2408_03865_amd/build.py).
    Without a path, the library named by LIB_PATH when the call is made, loaded once."""
    global _lib, _lib_path
    if path is None:
        path = LIB_PATH
    if _lib is not None and path == _lib_path:
        return _lib
    if not os.path.exists(path):
        raise FileNotFoundError(f"{path} is missing; build it with `python paper_2408_03865_amd/build.py`")
    # One HIP runtime per process: torch ships its own libamdhip64.so.7, and the library's
    # dependency of that name resolves to torch's copy only when torch is loaded first.
    # The other way round the process holds two runtimes, and launches on torch's streams
    # fail.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    lib.packmamba_abi_version.restype = ctypes.c_int
    lib.packmamba_status_string.argtypes = [ctypes.c_int]
    lib.packmamba_status_string.restype = ctypes.c_char_p
    lib.packmamba_causal_conv1d_fwd.argtypes = [vp] * 7 + [i64, i64, i64, i32, i32, i32, vp]
    lib.packmamba_causal_conv1d_bwd_workspace_size.argtypes = [i64, i64, i64, i32]
    lib.packmamba_causal_conv1d_bwd_workspace_size.restype = sz
    lib.packmamba_causal_conv1d_bwd.argtypes = [vp] * 12 + [sz, i64, i64, i64, i32, i32, i32, vp]
    lib.packmamba_causal_conv1d_bwd_noalloc.argtypes = [vp] * 11 + [i64, i64, i64, i32, i32, i32, vp]
    lib.packmamba_selective_scan_fwd_saved_states_size.argtypes = [i64, i64, i64, i32]
    lib.packmamba_selective_scan_fwd_saved_states_size.restype = sz
    lib.packmamba_selective_scan_fwd_workspace_size.argtypes = [i64, i64, i64, i32]
    lib.packmamba_selective_scan_fwd_workspace_size.restype = sz
    lib.packmamba_selective_scan_fwd.argtypes = [vp] * 8 + [i32] + [vp] * 6 + [sz, i64, i64, i64, i32, i32, vp]
    lib.packmamba_selective_scan_bwd_workspace_size.argtypes = [i64, i64, i64, i32]
    lib.packmamba_selective_scan_bwd_workspace_size.restype = sz
    lib.packmamba_selective_scan_bwd.argtypes = ([vp] * 8 + [i32] + [vp] * 15 + [sz, i64, i64, i64, i32, i32, vp])
    lib.packmamba_check_position_indices.argtypes = [vp, i64, i64, i32, vp, vp]
    lib.packmamba_pack_plan.argtypes = [vp, i64, i64, i32, i64, vp, i64, vp, vp]
    lib.packmamba_pack_positions.argtypes = [vp, i64, i64, i64, vp]
    lib.packmamba_rmsnorm_fwd.argtypes = [vp, vp, ctypes.c_float, vp, vp, i64, i64, i64, i32, vp]
    lib.packmamba_rmsnorm_bwd_workspace_size.argtypes = [i64, i64, i64]
    lib.packmamba_rmsnorm_bwd_workspace_size.restype = sz
    lib.packmamba_rmsnorm_bwd.argtypes = [vp] * 8 + [sz, i64, i64, i64, i32, vp]
    for name in ("packmamba_pack_plan", "packmamba_pack_positions", "packmamba_causal_conv1d_fwd",
                 "packmamba_causal_conv1d_bwd", "packmamba_causal_conv1d_bwd_noalloc",
                 "packmamba_selective_scan_fwd", "packmamba_selective_scan_bwd",
                 "packmamba_check_position_indices", "packmamba_rmsnorm_fwd", "packmamba_rmsnorm_bwd"):
        getattr(lib, name).restype = ctypes.c_int
    if lib.packmamba_abi_version() != ABI_VERSION:
        raise RuntimeError("libpackmamba ABI version mismatch")
    if path == LIB_PATH:
        _lib, _lib_path = lib, path
    return lib


def check(fn: str, status: int) -> None:
    if status != 0:
        text = load().packmamba_status_string(status).decode()
        raise PackMambaError(fn, status, text)
