"""The C-ABI library on the CPU: it loads, exports every declared symbol, and rejects bad
arguments before anything is enqueued (no GPU needed; skipped where a GPU is visible so
that fake pointers can never reach a kernel)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "packmamba.h")


def _lib():
    from paper_2408_03865_amd import _lib as L
    if not os.path.exists(L.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return L.load()


def test_exports_every_declared_symbol():
    from paper_2408_03865_amd import _lib as L
    names = set(re.findall(r"\b(packmamba_\w+)\s*\(", open(HEADER).read()))
    assert names == set(L.EXPORTS), names ^ set(L.EXPORTS)
    lib = _lib()
    for n in names:
        assert hasattr(lib, n), n
    assert lib.packmamba_abi_version() == 6


def test_status_strings():
    lib = _lib()
    for s in range(8):
        assert lib.packmamba_status_string(s)
        assert b"unknown" not in lib.packmamba_status_string(s)
    assert b"unknown" in lib.packmamba_status_string(99)


def test_sizes():
    lib = _lib()
    # chunk states, then the dz factor (rows padded to 256 tokens) from the next multiple of 256 bytes
    assert lib.packmamba_selective_scan_fwd_saved_states_size(8, 4096, 4096, 16) == \
        8 * 4096 * 32 * 16 * 4 + 8 * 4096 * 4096 * 4
    assert lib.packmamba_selective_scan_fwd_saved_states_size(1, 1, 129, 16) == 256 + 1024   # row padded to 256 tokens
    assert lib.packmamba_selective_scan_fwd_saved_states_size(1, 1, 129, 8) == 0
    assert lib.packmamba_causal_conv1d_bwd_workspace_size(2, 3, 5, 4) >= 2 * 3 * 5 * 4
    assert lib.packmamba_causal_conv1d_bwd_workspace_size(2, 3, 5, 5) == 0
    assert lib.packmamba_selective_scan_bwd_workspace_size(8, 4096, 4096, 16) > 0
    assert lib.packmamba_selective_scan_bwd_workspace_size(0, 4096, 4096, 16) == 0
    # forward workspace: only for shapes whose rows are split into segments
    assert lib.packmamba_selective_scan_fwd_workspace_size(8, 4096, 4096, 16) == 0
    assert lib.packmamba_selective_scan_fwd_workspace_size(1, 2048, 256, 16) == 0      # one 256-token unit
    assert lib.packmamba_selective_scan_fwd_workspace_size(1, 2048, 65536, 16) >= 1 * 2048 * 6 * 16 * 12   # 6 segments
    assert lib.packmamba_selective_scan_fwd_workspace_size(0, 2048, 65536, 16) == 0
    assert (lib.packmamba_selective_scan_bwd_workspace_size(1, 2048, 65536, 16)
            > lib.packmamba_selective_scan_fwd_workspace_size(1, 2048, 65536, 16))


def test_segment_rule():
    """The Python mirror of the segment rule (used by tests and reports) matches the
    workspace the library asks for."""
    import paper_2408_03865_amd as P
    lib = _lib()
    for shape in [(8, 4096, 4096), (8, 5120, 4096), (4, 1536, 2048), (2, 2048, 8192), (1, 2048, 65536),
                  (1, 64, 256), (1, 64, 257), (1, 16, 100000), (3, 700, 3000), (47, 16, 512),
                  (24, 16, 4096), (40, 16, 4096)]:
        b, d, _ = shape
        nf, nb = P.segments(*shape, direction="fwd"), P.segments(*shape)
        assert nf <= nb, shape                      # the backward's workspace covers the forward's plan
        ws = lib.packmamba_selective_scan_fwd_workspace_size(*shape, 16)
        assert (nf > 1) == (ws > 0), shape
        if nf > 1:
            assert ws >= b * d * nf * 16 * 12, shape
        wsb = lib.packmamba_selective_scan_bwd_workspace_size(*shape, 16)
        if nb > 1:
            assert wsb >= b * d * nb * 16 * 12, shape
    assert P.segments(8, 4096, 4096) == 1
    assert P.segments(1, 2048, 65536) == 12 and P.segments(1, 2048, 65536, "fwd") == 6
    assert P.segments(2, 2048, 8192) == 6 and P.segments(2, 2048, 8192, "fwd") == 3
    assert P.segments(4, 1536, 2048) == 4 and P.segments(4, 1536, 2048, "fwd") == 1   # 384 blocks
    assert P.segments(500, 16, 4096) == 4 and P.segments(500, 16, 4096, "fwd") == 1   # forward unsplit


def _gpu_visible():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.mark.skipif(_gpu_visible(), reason="fake pointers are only passed where no GPU exists")
def test_argument_errors_before_launch():
    lib = _lib()
    P = 0x10000          # fake, aligned; every case below must fail validation first
    U = 0x10008          # fake, misaligned
    conv = lib.packmamba_causal_conv1d_fwd
    # x, w, bias, pos, initial_x, out, final_x, batch, dim, seqlen, width, dtype, silu, stream
    assert conv(None, P, None, P, None, P, None, 1, 1, 8, 4, 0, 1, None) == 1     # x NULL
    assert conv(P, P, None, P, None, P, None, 0, 1, 8, 4, 0, 1, None) == 2        # batch 0
    assert conv(P, P, None, P, None, P, None, 1, 1, -3, 4, 0, 1, None) == 2       # seqlen < 0
    assert conv(P, P, None, P, None, P, None, 1, 1, 1 << 40, 4, 0, 1, None) == 2  # too large
    assert conv(P, P, None, P, None, P, None, 1, 1, 8, 5, 0, 1, None) == 3        # width 5
    assert conv(P, P, None, P, None, P, None, 1, 1, 8, 1, 0, 1, None) == 3        # width 1
    assert conv(P, P, None, P, None, P, None, 1, 1, 8, 4, 7, 1, None) == 3        # dtype
    assert conv(U, P, None, P, None, P, None, 1, 1, 8, 4, 0, 1, None) == 4        # misaligned x
    assert conv(P, P, None, P, U, P, None, 1, 1, 8, 4, 0, 1, None) == 4           # misaligned initial_x
    cbwd = lib.packmamba_causal_conv1d_bwd
    # x, w, bias, pos, initial_x, dout, dfinal_x, dx, dw, dbias, dinitial_x, ws, ws_bytes, ...
    assert cbwd(P, P, P, P, None, P, None, P, P, None, None, P, 1 << 20, 1, 1, 8, 4, 0, 1, None) == 1  # bias without dbias
    assert cbwd(P, P, None, P, P, P, None, P, P, None, None, P, 1 << 20, 1, 1, 8, 4, 0, 1, None) == 1  # initial_x without dinitial_x
    assert cbwd(P, P, None, P, None, P, None, P, P, None, P, P, 1 << 20, 1, 1, 8, 4, 0, 1, None) == 1  # dinitial_x without initial_x
    assert cbwd(P, P, None, P, None, P, None, P, P, None, None, P, 1, 1, 1, 8, 4, 0, 1, None) == 5     # workspace small
    assert cbwd(P, P, None, P, None, P, None, P, P, None, None, None, 1 << 20, 1, 1, 8, 4, 0, 1, None) == 5
    # the no-allocation variant: the same argument errors, and shapes beyond its fixed scratch
    na = lib.packmamba_causal_conv1d_bwd_noalloc
    # x, w, bias, pos, initial_x, dout, dfinal_x, dx, dw, dbias, dinitial_x, batch, dim, seqlen, width, dtype, silu, stream
    assert na(None, P, None, P, None, P, None, P, P, None, None, 1, 1, 8, 4, 0, 1, None) == 1
    assert na(P, P, P, P, None, P, None, P, P, None, None, 1, 1, 8, 4, 0, 1, None) == 1       # bias without dbias
    assert na(P, P, None, P, None, P, None, P, P, None, None, 0, 1, 8, 4, 0, 1, None) == 2
    assert na(P, P, None, P, None, P, None, P, P, None, None, 1, 1, 8, 5, 0, 1, None) == 3
    assert na(P, P, None, P, None, P, None, U, P, None, None, 1, 1, 8, 4, 0, 1, None) == 4
    big = (8, 1 << 17, 8)   # 8 x 131072 x 5 partial floats = 20 MiB > 16 MiB
    assert lib.packmamba_causal_conv1d_bwd_workspace_size(*big, 4) > (16 << 20)
    assert na(P, P, None, P, None, P, None, P, P, None, None, *big, 4, 0, 1, None) == 7
    assert lib.packmamba_causal_conv1d_bwd_workspace_size(8, 4096, 4096, 4) <= (16 << 20)
    fwd = lib.packmamba_selective_scan_fwd
    # u, delta, A, B, C, D, z, delta_bias, softplus, pos, initial_state, out, final_state, states,
    # ws, ws_bytes, batch, dim, seqlen, dstate, dtype, stream
    args = [P, P, P, P, P, None, None, None, 1, P, None, P, None, None, None, 0, 1, 1, 8, 16, 1, None]
    a = list(args); a[0] = None
    assert fwd(*a) == 1
    a = list(args); a[11] = None                                            # no out, states or final state
    assert fwd(*a) == 1
    a = list(args); a[19] = 8                                               # dstate 8
    assert fwd(*a) == 3
    a = list(args); a[6] = U                                                # misaligned z
    assert fwd(*a) == 4
    a = list(args); a[12] = U                                               # misaligned final_state
    assert fwd(*a) == 4
    a = list(args); a[16] = 70000                                           # batch too large
    assert fwd(*a) == 2
    a = list(args); a[17] = 16; a[18] = 65536                               # split rows need a workspace
    assert fwd(*a) == 5
    a[14] = P; a[15] = 64
    assert fwd(*a) == 5
    a[14] = U; a[15] = 1 << 30
    assert fwd(*a) == 4
    bwd = lib.packmamba_selective_scan_bwd
    # u, delta, A, B, C, D, z, delta_bias, softplus, pos, initial_state, dout, dfinal_state, states,
    # du, ddelta, dA, dB, dC, dD, dz, ddelta_bias, dinitial_state, ws, ws_bytes, batch, dim, seqlen,
    # dstate, dtype, stream
    bargs = [P, P, P, P, P, P, None, None, 1, P, None, P, None, None, P, P, P, P, P, P, None, None, None,
             P, 1 << 40, 1, 1, 8, 16, 1, None]
    a = list(bargs); a[19] = None                                           # D without dD
    assert bwd(*a) == 1
    a = list(bargs); a[20] = P                                              # dz without z
    assert bwd(*a) == 1
    a = list(bargs); a[10] = P                                              # initial_state without its gradient
    assert bwd(*a) == 1
    a = list(bargs); a[22] = P                                              # dinitial_state without initial_state
    assert bwd(*a) == 1
    a = list(bargs); a[24] = 16                                             # workspace too small
    assert bwd(*a) == 5
    a = list(bargs); a[28] = 32
    assert bwd(*a) == 3
    assert lib.packmamba_check_position_indices(None, 1, 8, 0, P, None) == 1
    assert lib.packmamba_check_position_indices(U, 1, 8, 1, P, None) == 4
    # RMSNorm
    nf, nb = lib.packmamba_rmsnorm_fwd, lib.packmamba_rmsnorm_bwd
    assert nf(None, P, 1e-5, P, P, 1, 4, 8, 0, None) == 1
    assert nf(P, P, 1e-5, P, None, 1, 4, 8, 0, None) == 1
    assert nf(P, P, 1e-5, P, P, 0, 4, 8, 0, None) == 2
    assert nf(P, P, -1.0, P, P, 1, 4, 8, 0, None) == 2
    assert nf(P, P, float("nan"), P, P, 1, 4, 8, 0, None) == 2
    assert nf(P, P, 1e-5, P, P, 1, 4, 8, 9, None) == 3
    assert nf(U, P, 1e-5, P, P, 1, 4, 8, 0, None) == 4
    ws = lib.packmamba_rmsnorm_bwd_workspace_size(2, 4, 100)
    assert ws >= 2 * 2 * 4 * 4 and lib.packmamba_rmsnorm_bwd_workspace_size(0, 4, 100) == 0
    assert nb(P, P, P, P, None, P, None, P, ws, 2, 4, 100, 0, None) == 1                # no dweight
    assert nb(P, P, P, P, None, P, P, P, ws - 1, 2, 4, 100, 0, None) == 5
    assert nb(P, P, P, P, U, P, P, P, ws, 2, 4, 100, 0, None) == 4                     # dresidual
    assert nb(P, P, P, P, None, P, P, P, ws, 2, 4, 100, 5, None) == 3


def test_one_hip_runtime_per_process():
    """Loading the library first must not put a second HIP runtime next to torch's own:
    launches on torch's streams fail in such a process."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = ("import sys; sys.path.insert(0, %r)\n"
            "from paper_2408_03865_amd import _lib\n"
            "_lib.load()\n"
            "import torch\n"
            "maps = open('/proc/self/maps').read().splitlines()\n"
            "print(len({l.split()[-1] for l in maps if 'libamdhip64' in l}))\n") % root
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip().splitlines()[-1] == "1"


def test_load_follows_lib_path(tmp_path):
    """load() without a path returns the library that LIB_PATH names when it is called,
    also after LIB_PATH has changed (each file is loaded once)."""
    import shutil
    from paper_2408_03865_amd import _lib as L
    first = _lib()
    old = L.LIB_PATH
    copy = tmp_path / "libpackmamba_copy.so"
    shutil.copy(old, copy)
    try:
        L.LIB_PATH = str(copy)
        second = L.load()
        assert second._name == str(copy) and second is not first
        assert L.load() is second
    finally:
        L.LIB_PATH = old
    assert L.load()._name == old
