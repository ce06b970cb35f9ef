"""GPU parity of the packed Mamba block (paper_2408_03865_amd/block.py): forward and every
gradient against the fp64 block oracle (fp32 path; the bf16 path re-rounds every GEMM
output, so its block chain is not compared with an unrounded oracle chain -- the
per-operator bf16 parity covers the kernels), and packing-unpacking invariance on the GPU."""
import numpy as np
import pytest

import workloads as W
from gpu_common import TOL, assert_close, f32, host, i32, note

pytestmark = pytest.mark.gpu

DIMS = dict(d_model=64, Dn=128, N=16, R=8, Wd=4)


def _params(d_model, Dn, N, R, Wd, seed):
    rng = np.random.default_rng(seed)
    s = lambda *sh: rng.standard_normal(sh) / np.sqrt(sh[-1])  # noqa: E731
    return dict(norm_w=rng.uniform(0.5, 1.5, d_model), W_in=s(2 * Dn, d_model),
                conv_w=rng.uniform(-0.5, 0.5, (Dn, Wd)), conv_b=rng.uniform(-0.5, 0.5, Dn),
                W_x=s(R + 2 * N, Dn), W_dt=s(Dn, R), dt_bias=rng.uniform(-4.0, -1.0, Dn),
                A=-np.exp(rng.normal(0, 0.5, (Dn, N))), D=rng.standard_normal(Dn), W_out=s(d_model, Dn))


def _to_gpu(p):
    return {k: f32(v.astype(np.float32)) for k, v in p.items()}


def _cast(p):
    """The values the GPU sees (fp32), back in fp64 for the oracle."""
    return {k: v.astype(np.float32).astype(np.float64) for k, v in p.items()}


@pytest.mark.parametrize("shape", [(2, 300), (1, 1025), (3, 64)], ids=lambda s: f"{s[0]}x{s[1]}")
def test_block_matches_oracle_f32(shape):
    import torch
    import oracle.block as OB
    import paper_2408_03865_amd.block as BK
    batch, L = shape
    note(f"block {shape}")
    p = _params(**DIMS, seed=batch * 7 + L)
    rng = np.random.default_rng(L)
    rows = W.draw_row_lengths(("lognormal", 3.5, 1.0, 1, L), rng, batch, L)
    pos = W.positions_from_lengths(rows, L)
    x = rng.standard_normal((batch, DIMS["d_model"], L)).astype(np.float32)
    dout = rng.standard_normal((batch, DIMS["d_model"], L)).astype(np.float32)
    gp = _to_gpu(p)
    out, ctx = BK.block_forward(f32(x), i32(pos), gp)
    g = BK.block_backward(f32(dout), ctx, gp)
    torch.cuda.synchronize()
    q = _cast(p)
    ref_out = OB.block_fwd(x.astype(np.float64), pos, q)
    ref = OB.block_bwd(x.astype(np.float64), pos, q, dout.astype(np.float64))
    tol = TOL["f32"]
    assert_close("block out", host(out), ref_out, tol)
    for k in ref:
        assert_close(f"block d{k}", host(g[k]), ref[k], tol)


def test_block_pui_on_gpu():
    """Packed rows through the GPU block == each sequence's own GPU block run (fp32)."""
    import torch
    import paper_2408_03865_amd.block as BK
    p = _to_gpu(_params(**DIMS, seed=5))
    rows = [[37, 1, 90, 3, 125], [256]]
    L = 256
    rng = np.random.default_rng(6)
    x = rng.standard_normal((2, DIMS["d_model"], L)).astype(np.float32)
    dout = rng.standard_normal((2, DIMS["d_model"], L)).astype(np.float32)
    pos = W.positions_from_lengths(rows, L)
    out, ctx = BK.block_forward(f32(x), i32(pos), p)
    g = BK.block_backward(f32(dout), ctx, p)
    acc = {k: 0.0 for k in g if k != "x"}
    for b, row in enumerate(rows):
        s = 0
        for n in row:
            sl = slice(s, s + n)
            o1, c1 = BK.block_forward(f32(x[b:b + 1, :, sl]), i32(np.arange(n, dtype=np.int32)[None]), p)
            g1 = BK.block_backward(f32(dout[b:b + 1, :, sl]), c1, p)
            assert_close(f"pui out {b},{s}", host(out[b:b + 1, :, sl]), host(o1), TOL["f32"])
            assert_close(f"pui dx {b},{s}", host(g["x"][b:b + 1, :, sl]), host(g1["x"]), TOL["f32"])
            for k in acc:
                acc[k] = acc[k] + host(g1[k])
            s += n
    torch.cuda.synchronize()
    for k in acc:
        assert_close(f"pui d{k}", host(g[k]), acc[k], TOL["f32"])
