"""Helpers shared by the GPU tests: device transfer, the GPU call chain and comparisons."""
from __future__ import annotations

import sys
from typing import Dict

import numpy as np

import workloads as W

TOL = {"f32": 1e-4, "bf16": 2e-3}


def torch():
    import torch as t
    return t


def dev():
    return torch().device("cuda:0")


def act(a: np.ndarray, dtype: str):
    """Activation tensor on the GPU in the path dtype (values are already representable)."""
    t = torch().from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    if dtype == "bf16":
        t = t.to(torch().bfloat16)
    return t.to(dev())


def f32(a):
    if a is None:
        return None
    return torch().from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev())


def i32(a):
    return torch().from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev())


def host(t) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


def note(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def assert_close(name: str, got: np.ndarray, ref: np.ndarray, tol: float) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    err = np.abs(got - ref) / (1.0 + np.abs(ref))
    i = int(np.argmax(err))
    m = float(err.flat[i])
    idx = np.unravel_index(i, err.shape)
    assert m <= tol, f"{name}: max |err|/(1+|ref|) = {m:.3e} > {tol:.1e} at {idx}: got {got[idx]!r} ref {ref[idx]!r}"
    return m


def gpu_inputs(d: Dict[str, np.ndarray], dtype: str, general: bool = False):
    g = {k: act(d[k], dtype) for k in W.ACTIVATIONS}
    for k in ("A", "D", "delta_bias", "w", "bias"):
        g[k] = f32(d[k])
    g["pos"] = i32(d["pos"])
    return g


def run_gpu(g, out_f32: bool = False, states: bool = True, opts=None):
    """conv fwd/bwd on (x, dout) and scan fwd/bwd on (u, delta, z, B, C, dout)."""
    import paper_2408_03865_amd as P
    o = dict(D=g["D"], z=g["z"], delta_bias=g["delta_bias"], softplus=True, bias=g["bias"],
             silu=True)
    if opts:
        o.update(opts)
    r = {}
    r["conv_out"] = P.causal_conv1d_fwd(g["x"], g["w"], o["bias"], g["pos"], silu=o["silu"], out_f32=out_f32)
    r["dx"], r["dw"], r["dbias"] = P.causal_conv1d_bwd(g["x"], g["w"], o["bias"], g["pos"], g["dout"],
                                                       silu=o["silu"], out_f32=out_f32)
    out, st = P.selective_scan_fwd(g["u"], g["delta"], g["A"], g["B"], g["C"], o["D"], o["z"],
                                   o["delta_bias"], o["softplus"], g["pos"], return_states=True,
                                   out_f32=out_f32)
    r["out"], r["states"] = out, st
    r.update(P.selective_scan_bwd(g["u"], g["delta"], g["A"], g["B"], g["C"], o["D"], o["z"],
                                  o["delta_bias"], o["softplus"], g["pos"], g["dout"],
                                  saved_states=st if states else None, out_f32=out_f32))
    torch().cuda.synchronize()
    return r


def oracle_run(d, sl_b=slice(None), sl_d=slice(None), opts=None):
    """Oracle fwd/bwd of both operators on the sub-problem (batch rows sl_b, channels sl_d)."""
    import oracle as O
    o = dict(D=d["D"], z=d["z"], delta_bias=d["delta_bias"], softplus=True, bias=d["bias"], silu=True)
    if opts:
        o.update(opts)

    def a(k):
        return d[k][sl_b][:, sl_d]

    def p(v):
        return None if v is None else v[sl_d]

    r = {}
    r["conv_out"] = O.conv1d_fwd(a("x"), d["w"][sl_d], p(o["bias"]), d["pos"][sl_b], silu=o["silu"])
    cg = O.conv1d_bwd(a("x"), d["w"][sl_d], p(o["bias"]), d["pos"][sl_b], a("dout"), silu=o["silu"])
    r["dx"], r["dw"], r["dbias"] = cg["dx"], cg["dw"], cg["dbias"]
    z = None if o["z"] is None else o["z"][sl_b][:, sl_d]
    args = dict(u=a("u"), delta=a("delta"), A=d["A"][sl_d], B=d["B"][sl_b], C=d["C"][sl_b],
                D=p(o["D"]), z=z, delta_bias=p(o["delta_bias"]), delta_softplus=o["softplus"],
                pos=d["pos"][sl_b])
    r["out"] = O.scan_fwd(**args)
    r.update(O.scan_bwd(**args, dout=a("dout")))
    return r


PER_TOKEN = ("conv_out", "dx", "out", "du", "ddelta", "dz")
PER_CHANNEL = ("dw", "dbias", "dA", "dD", "ddelta_bias")
PER_B = ("dB", "dC")


def compare(gr, ref, tol, keys, sl_b=slice(None), sl_d=slice(None), label=""):
    worst = {}
    for k in keys:
        if ref.get(k) is None:
            assert gr.get(k) is None, k
            continue
        t = gr[k]
        if k in PER_TOKEN:
            got = host(t[sl_b][:, sl_d])
        elif k in PER_CHANNEL:
            got = host(t[sl_d])
        elif k in PER_B:
            got = host(t[sl_b])
        else:
            got = host(t)
        worst[k] = assert_close(f"{label}{k}", got, ref[k], tol)
    note(f"{label} worst scaled errors: " + ", ".join(f"{k}={v:.2e}" for k, v in worst.items()))
    return worst


BF16_OUT = ("conv_out", "dx", "out", "du", "ddelta", "dz")
# fp32-typed outputs (the saved-states buffer is opaque and has unwritten alignment gaps
# at some shapes, so it is not compared as a whole)
F32_ALWAYS = ("dw", "dbias", "dA", "dD", "ddelta_bias", "dB", "dC")


def check_bf16_rounding(r_bf, r_f32, label, keys=BF16_OUT, same=F32_ALWAYS):
    """The bf16-output run (dtype code 1) equals the round-to-nearest-even of the fp32-output
    run (dtype code 2) on every element, and the fp32-typed outputs of both are identical."""
    for k in keys:
        if r_f32.get(k) is None:
            assert r_bf.get(k) is None, k
            continue
        a, b = bf16_bits_of(r_bf[k]), rne_bf16(r_f32[k])
        bad = np.count_nonzero(a != b)
        assert bad == 0, f"{label}{k}: {bad} bf16 outputs differ from RNE of the fp32 outputs"
    for k in same:
        if r_f32.get(k) is None:
            continue
        assert np.array_equal(host(r_bf[k]), host(r_f32[k])), f"{label}{k} differs between dtype codes"


def rne_bf16(t) -> np.ndarray:
    """bf16 bit patterns of the round-to-nearest-even of an fp32 tensor."""
    return W.bf16_bits(t.float().cpu().numpy())


def bf16_bits_of(t) -> np.ndarray:
    return t.contiguous().view(torch().int16).cpu().numpy().view(np.uint16)
