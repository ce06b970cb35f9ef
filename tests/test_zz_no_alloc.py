"""The no-allocation conv1d backward (packmamba_causal_conv1d_bwd_noalloc), called through
the C ABI, against the workspace entry point packmamba_causal_conv1d_bwd on the same
inputs: every output equal bit for bit (the same kernels, with the partials in the
library's fixed scratch instead of a workspace), and both within the bound of the
oracle.  Two calls in a row, the second on a smaller input, so that the second call
runs over the scratch contents the first left behind."""
import ctypes

import numpy as np
import pytest

import workloads as W
from gpu_common import TOL, assert_close, gpu_inputs, host, note, torch

pytestmark = pytest.mark.gpu


def _call_pair(g, dtype, width, states, seed):
    import oracle as O
    from paper_2408_03865_amd import _lib
    lib = _lib.load()
    t = torch()
    x, w, bias, pos, dout = g["x"], g["w"][:, :width].contiguous(), g["bias"], g["pos"], g["dout"]
    Nb, Dn, L = x.shape
    code = _lib.F32 if dtype == "f32" else _lib.BF16
    gen = t.Generator(device="cuda:0").manual_seed(seed)
    xi = dxf = None
    if states:
        xi = t.randn((Nb, Dn, width - 1), generator=gen, device="cuda:0").to(x.dtype)
        dxf = t.randn((Nb, Dn, width - 1), generator=gen, device="cuda:0").to(x.dtype)
    P = lambda v: None if v is None else v.data_ptr()  # noqa: E731
    stream = t.cuda.current_stream().cuda_stream
    outs = []
    for noalloc in (False, True):
        dx = t.full_like(x, float("nan"))
        dw = t.full_like(w, float("nan"))
        db = t.full_like(bias, float("nan"))
        dxi = t.full_like(xi, float("nan")) if states else None
        if noalloc:
            st = lib.packmamba_causal_conv1d_bwd_noalloc(
                P(x), P(w), P(bias), P(pos), P(xi), P(dout), P(dxf), P(dx), P(dw), P(db), P(dxi),
                Nb, Dn, L, width, code, 1, stream)
        else:
            need = lib.packmamba_causal_conv1d_bwd_workspace_size(Nb, Dn, L, width)
            ws = t.full((need // 4,), float("nan"), dtype=t.float32, device="cuda:0")
            st = lib.packmamba_causal_conv1d_bwd(
                P(x), P(w), P(bias), P(pos), P(xi), P(dout), P(dxf), P(dx), P(dw), P(db), P(dxi),
                P(ws), need, Nb, Dn, L, width, code, 1, stream)
        _lib.check("conv1d_bwd" + ("_noalloc" if noalloc else ""), st)
        t.cuda.synchronize()
        outs.append({"dx": dx, "dw": dw, "dbias": db, "dxinit": dxi})
    ref, got = outs
    for k, v in ref.items():
        if v is None:
            continue
        assert t.equal(got[k], v), f"noalloc {k} differs from the workspace entry point"
    # both against the oracle (bf16: the dx comparison is on bf16-rounded outputs, so
    # only the fp32 parameter gradients are held to the bound here)
    o = O.conv1d_bwd(host(x), host(w), host(bias), host(pos).astype(np.int32), host(dout), silu=True,
                     xinit=None if xi is None else host(xi), dxfinal=None if dxf is None else host(dxf))
    tol = TOL[dtype]
    keys = ("dx", "dw", "dbias", "dxinit") if dtype == "f32" else ("dw", "dbias")
    for k in keys:
        if o.get(k) is not None:
            assert_close(f"noalloc {k}", host(got[k]), o[k], tol)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_matches_workspace_entry_point(dtype):
    for i, (shape, width, states) in enumerate([((3, 70, 1000), 4, True), ((2, 17, 129), 3, False)]):
        batch, dim, seqlen = shape
        note(f"noalloc conv1d bwd call {i}: {shape} width {width} {dtype} states={states}")
        cfg = W.Config("noalloc", "noalloc", batch, seqlen, dim, 16, 4, dtype,
                       ("lognormal", 3.0, 1.0, 1, seqlen), 8800 + i)
        d = W.make_inputs(cfg, variant="general")
        _call_pair(gpu_inputs(d, dtype), dtype, width, states, seed=i)


def test_noalloc_rejects_beyond_scratch():
    from paper_2408_03865_amd import _lib
    lib = _lib.load()
    t = torch()
    x = t.zeros(16, device="cuda:0")
    p = x.data_ptr()
    big = (8, 1 << 17, 8)
    st = lib.packmamba_causal_conv1d_bwd_noalloc(p, p, None, p, None, p, None, p, p, None, None, *big, 4, 0, 1,
                                                 t.cuda.current_stream().cuda_stream)
    assert st == 7, st
