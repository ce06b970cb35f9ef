"""The hand-derived integer fixture of tests/golden/probe_row12.json: one packed row of
12 tokens (sequences of lengths 1, 4, 2, 5), conv tap-mask probe (Alg. 1) and scan
reset probe (Alg. 2, §3.4).  The oracle must reproduce every value exactly on the CPU,
and the HIP kernels on the GPU, in fp32 and bf16 (all values are small integers,
exact in both)."""
import json
import os

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
FIX = json.load(open(os.path.join(HERE, "golden", "probe_row12.json")))


def _setup():
    pos = np.array([FIX["positions"]], dtype=np.int32)
    Dn, L, N, W = FIX["dim"], pos.shape[1], 16, 4
    ones = np.ones((1, Dn, L))
    w = np.tile(np.array([1.0, 2.0, 4.0, 8.0]), (Dn, 1))
    e0 = np.zeros((1, N, L))
    e0[:, 0] = 1.0
    return pos, Dn, L, N, W, ones, w, e0


def _check(conv_out, conv_g, scan_out, scan_g):
    c, s = FIX["conv"], FIX["scan"]
    for d in range(FIX["dim"]):
        assert np.array_equal(conv_out[0, d], c["out"]), ("conv out", conv_out[0, d])
        assert np.array_equal(conv_g["dx"][0, d], c["dx"]), ("conv dx", conv_g["dx"][0, d])
        assert np.array_equal(conv_g["dw"][d], c["dweight"]), ("dweight", conv_g["dw"][d])
        assert conv_g["db"][d] == c["dbias"]
        assert np.array_equal(scan_out[0, d], s["y"]), ("scan y", scan_out[0, d])
        assert np.array_equal(scan_g["du"][0, d], s["du"])
        assert np.array_equal(scan_g["ddelta"][0, d], s["ddelta"])
        assert scan_g["dA"][d, 0] == s["dA_state0"] and not scan_g["dA"][d, 1:].any()
        assert scan_g["dD"][d] == s["dD"] and scan_g["ddelta_bias"][d] == s["ddelta_bias"]
    assert np.array_equal(scan_g["dB"][0, 0], s["dB_state0"]) and not scan_g["dB"][0, 1:].any()
    assert np.array_equal(scan_g["dC"][0, 0], s["dC_state0"]) and not scan_g["dC"][0, 1:].any()


def test_oracle_matches_golden():
    import oracle as O
    pos, Dn, L, N, W, ones, w, e0 = _setup()
    zb = np.zeros(Dn)
    out = O.conv1d_fwd(ones, w, zb, pos, silu=False)
    cg = O.conv1d_bwd(ones, w, zb, pos, ones, silu=False)
    args = dict(u=ones, delta=ones, A=np.zeros((Dn, N)), B=e0, C=e0, D=np.zeros(Dn), z=None,
                delta_bias=np.zeros(Dn), delta_softplus=False, pos=pos)
    y = O.scan_fwd(**args)
    sg = O.scan_bwd(**args, dout=ones)
    _check(out, {"dx": cg["dx"], "dw": cg["dw"], "db": cg["dbias"]}, y, sg)


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_kernels_match_golden(dtype):
    import torch
    import paper_2408_03865_amd as P
    from gpu_common import f32, host, i32, note
    note(f"golden probe row, {dtype}")
    pos, Dn, L, N, W, ones, w, e0 = _setup()
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32

    def act(a):
        return torch.from_numpy(a.astype(np.float32)).to(tdt).to("cuda:0")

    x, e0d, p = act(ones), act(e0), i32(pos)
    wd, zb = f32(w), f32(np.zeros(Dn))
    out = P.causal_conv1d_fwd(x, wd, zb, p, silu=False, out_f32=True)
    dx, dw, db = P.causal_conv1d_bwd(x, wd, zb, p, x, silu=False, out_f32=True)
    A, D, dbias = f32(np.zeros((Dn, N))), f32(np.zeros(Dn)), f32(np.zeros(Dn))
    y, st = P.selective_scan_fwd(x, x, A, e0d, e0d, D, None, dbias, False, p, return_states=True,
                                 out_f32=True)
    g = P.selective_scan_bwd(x, x, A, e0d, e0d, D, None, dbias, False, p, x, saved_states=st, out_f32=True)
    torch.cuda.synchronize()
    sg = {k: host(v) for k, v in g.items() if v is not None}
    _check(host(out), {"dx": host(dx), "dw": host(dw), "db": host(db)}, host(y), sg)
