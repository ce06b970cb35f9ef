"""GPU parity of the RMSNorm kernels (the packed block's token-wise normalisation)
against the fp64 oracle of oracle/block.py, on the exact values the device sees:
forward output and rstd, backward dx (with and without a residual gradient) and
dweight; fp32 and bf16 inputs, ragged token counts (not multiples of the 8-token
vectors or the 64-token tiles) and feature counts that are not multiples of the
32 feature slices.  bf16 outputs are the fp32 results rounded once."""
import numpy as np
import pytest

from gpu_common import TOL, assert_close, f32, host, note

pytestmark = pytest.mark.gpu

SHAPES = [(2, 96, 200), (1, 40, 64), (3, 33, 1001), (1, 2048, 130)]


def _inputs(shape, seed):
    rng = np.random.default_rng(seed)
    b, d, L = shape
    x = rng.standard_normal(shape) * rng.uniform(0.2, 3.0, (b, 1, L))    # per-token scale
    g = rng.standard_normal(shape)
    res = rng.standard_normal(shape)
    w = rng.uniform(0.5, 1.5, d)
    return x, g, res, w


def _dev(a, dtype):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return (t.to(torch.bfloat16) if dtype == "bf16" else t).to("cuda:0")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_rmsnorm_matches_oracle(shape, dtype):
    import oracle.block as OB
    import paper_2408_03865_amd as P
    note(f"rmsnorm {shape} {dtype}")
    x, g, res, w = _inputs(shape, 11)
    xd, gd, rd, wd = _dev(x, dtype), _dev(g, dtype), _dev(res, dtype), f32(w)
    # the oracle sees the values the device holds
    x64, g64, r64 = host(xd), host(gd), host(rd)
    w64 = w.astype(np.float32).astype(np.float64)
    h, rstd = OB.rmsnorm(x64, w64)
    dx, dw = OB.rmsnorm_bwd(x64, w64, rstd, g64)
    out32 = dtype == "bf16"
    o, rs = P.rmsnorm_fwd(xd, wd, out_f32=out32)
    tol = TOL["f32"]
    assert_close("rstd", host(rs), rstd[:, 0, :], tol)
    assert_close("out", host(o), h, tol)
    dxg, dwg = P.rmsnorm_bwd(xd, wd, rs, gd, out_f32=out32)
    assert_close("dx", host(dxg), dx, tol)
    assert_close("dweight", host(dwg), dw, tol)
    dxr, dwr = P.rmsnorm_bwd(xd, wd, rs, gd, dresidual=rd, out_f32=out32)
    assert_close("dx + residual", host(dxr), dx + r64, tol)
    assert np.array_equal(host(dwr), host(dwg))
    if dtype == "bf16":
        # bf16 outputs: the fp32 values rounded once
        import torch
        ob, _ = P.rmsnorm_fwd(xd, wd)
        assert torch.equal(ob, o.to(torch.bfloat16))
        db, _ = P.rmsnorm_bwd(xd, wd, rs, gd, dresidual=rd)
        assert torch.equal(db, dxr.to(torch.bfloat16))


def test_rmsnorm_deterministic():
    import paper_2408_03865_amd as P
    x, g, _, w = _inputs((2, 300, 777), 5)
    xd, gd, wd = _dev(x, "bf16"), _dev(g, "bf16"), f32(w)
    o1, r1 = P.rmsnorm_fwd(xd, wd)
    o2, r2 = P.rmsnorm_fwd(xd, wd)
    d1, w1 = P.rmsnorm_bwd(xd, wd, r1, gd)
    d2, w2 = P.rmsnorm_bwd(xd, wd, r2, gd)
    for a, b in ((o1, o2), (r1, r2), (d1, d2), (w1, w2)):
        assert np.array_equal(host(a), host(b))
