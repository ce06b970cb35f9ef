"""Pins of the fp64 block oracle (oracle/block.py), CPU only: RMSNorm against torch's
rms_norm, packing-unpacking invariance of the whole block (§3.1: the composition of
PUI operators is PUI), and central finite differences of every block gradient."""
import numpy as np
import pytest

import oracle.block as OB
import workloads as W


def _params(d_model, Dn, N, R, Wd, seed):
    rng = np.random.default_rng(seed)
    s = lambda *sh: rng.standard_normal(sh) / np.sqrt(sh[-1])  # noqa: E731
    return dict(norm_w=rng.uniform(0.5, 1.5, d_model), W_in=s(2 * Dn, d_model),
                conv_w=rng.uniform(-0.5, 0.5, (Dn, Wd)), conv_b=rng.uniform(-0.5, 0.5, Dn),
                W_x=s(R + 2 * N, Dn), W_dt=s(Dn, R), dt_bias=rng.uniform(-2.0, -0.5, Dn),
                A=-np.exp(rng.normal(0, 0.5, (Dn, N))), D=rng.standard_normal(Dn), W_out=s(d_model, Dn))


def test_rmsnorm_matches_torch():
    import torch
    import torch.nn.functional as F
    rng = np.random.default_rng(0)
    x = rng.standard_normal((2, 8, 5))
    w = rng.uniform(0.5, 1.5, 8)
    h, _ = OB.rmsnorm(x, w)
    ref = F.rms_norm(torch.from_numpy(x).transpose(1, 2), (8,), torch.from_numpy(w), eps=OB.EPS)
    np.testing.assert_allclose(h, ref.transpose(1, 2).numpy(), rtol=1e-13, atol=1e-14)


def test_block_pui():
    """Packed block == each sequence's block run alone (outputs, input gradients); the
    parameter gradients are the sums over sequences."""
    p = _params(6, 8, 3, 2, 4, seed=1)
    rows = [[7, 1, 12, 4], [24]]
    L = 24
    rng = np.random.default_rng(2)
    x = rng.standard_normal((2, 6, L))
    dout = rng.standard_normal((2, 6, L))
    pos = W.positions_from_lengths(rows, L)
    out = OB.block_fwd(x, pos, p)
    g = OB.block_bwd(x, pos, p, dout)
    acc = {k: 0.0 for k in p}
    for b, row in enumerate(rows):
        s = 0
        for n in row:
            sl = slice(s, s + n)
            p1 = np.arange(n, dtype=np.int32)[None]
            o1 = OB.block_fwd(x[b:b + 1, :, sl], p1, p)
            g1 = OB.block_bwd(x[b:b + 1, :, sl], p1, p, dout[b:b + 1, :, sl])
            np.testing.assert_allclose(out[b:b + 1, :, sl], o1, rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(g["x"][b:b + 1, :, sl], g1["x"], rtol=1e-11, atol=1e-11)
            for k in p:
                acc[k] = acc[k] + g1[k]
            s += n
    for k in p:
        np.testing.assert_allclose(g[k], acc[k], rtol=1e-10, atol=1e-11, err_msg=k)


def test_block_finite_differences():
    p = _params(4, 6, 3, 2, 4, seed=3)
    rows = [[5, 1, 6]]
    L = 12
    rng = np.random.default_rng(4)
    x = rng.standard_normal((1, 4, L))
    dout = rng.standard_normal((1, 4, L))
    pos = W.positions_from_lengths(rows, L)
    g = OB.block_bwd(x, pos, p, dout)
    params = dict(p, x=x)

    def loss():
        return float(np.sum(dout * OB.block_fwd(params["x"], pos, {k: params[k] for k in p})))

    for k, arr in params.items():
        num = np.zeros_like(arr)
        it = np.nditer(arr, flags=["multi_index"])
        for _ in it:
            i = it.multi_index
            v = arr[i]
            eps = 1e-6 * max(1.0, abs(v))
            arr[i] = v + eps
            fp = loss()
            arr[i] = v - eps
            fm = loss()
            arr[i] = v
            num[i] = (fp - fm) / (2 * eps)
        err = np.abs(g[k] - num) / (1.0 + np.abs(num))
        assert err.max() < 1e-6, (k, float(err.max()))
