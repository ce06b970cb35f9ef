"""Bit-exact integer probes of the masks and resets, at every config's position indices.

With A = 0 (so exp(0) = 1 exactly), unit step without softplus, B = C = e_0 and
u = 1, the scan output is the position index plus one and, with dout = 1, du is
the number of tokens left in the sequence: any reset placed one token off, or a
state leaking across a start, changes an integer.  The conv probe uses taps
1, 2, 4, 8 so that every output is the bit mask of its live taps.  Expected
values come from the position indices alone (integer arithmetic), not the oracle.
"""
import numpy as np
import pytest

import workloads as W
from gpu_common import f32, host, i32, note, torch

pytestmark = pytest.mark.gpu

DIM = 32


def _pos(key):
    cfg = W.config(key)
    rng = np.random.Generator(np.random.PCG64(cfg.seed))
    rows = W.draw_row_lengths(cfg.lengths, rng, cfg.batch, cfg.seqlen)
    return cfg, W.positions_from_lengths(rows, cfg.seqlen)


def _remaining(pos):
    """tokens from l to the end of l's sequence (inclusive)"""
    Nb, L = pos.shape
    rem = np.zeros_like(pos, dtype=np.int64)
    for b in range(Nb):
        nxt = 0
        for l in range(L - 1, -1, -1):
            rem[b, l] = nxt + 1 if (l + 1 < L and pos[b, l + 1] != 0) else 1
            nxt = rem[b, l]
    return rem


def _act(a, dtype):
    t = torch().from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return (t.to(torch().bfloat16) if dtype != "f32" else t).to("cuda:0")


@pytest.mark.parametrize("key,out_f32", [("0", True), ("1", True), ("2", True), ("3", True),
                                         ("4a", True), ("4a", False), ("4b", True)])
def test_scan_probe(key, out_f32):
    import paper_2408_03865_amd as P
    cfg, pos = _pos(key)
    note(f"scan probe config {key} out_f32={out_f32}")
    Nb, L, N = cfg.batch, cfg.seqlen, cfg.dstate
    ones = np.ones((Nb, DIM, L), np.float32)
    e0 = np.zeros((Nb, N, L), np.float32)
    e0[:, 0, :] = 1
    u, dl, dout = _act(ones, cfg.dtype), _act(ones, cfg.dtype), _act(ones, cfg.dtype)
    B, C = _act(e0, cfg.dtype), _act(e0, cfg.dtype)
    A = f32(np.zeros((DIM, N)))
    p = i32(pos)
    out, st = P.selective_scan_fwd(u, dl, A, B, C, None, None, None, False, p, return_states=True,
                                   out_f32=out_f32)
    g = P.selective_scan_bwd(u, dl, A, B, C, None, None, None, False, p, dout, saved_states=st,
                             out_f32=out_f32)
    torch().cuda.synchronize()
    rem = _remaining(pos).astype(np.float64)
    want_y = np.broadcast_to((pos + 1)[:, None, :], (Nb, DIM, L))
    assert np.array_equal(host(out), want_y), "y != position index + 1"
    assert np.array_equal(host(g["du"]), np.broadcast_to(rem[:, None, :], (Nb, DIM, L))), "du != tokens left"
    assert np.array_equal(host(g["ddelta"]), np.broadcast_to(rem[:, None, :], (Nb, DIM, L))), "ddelta"
    dB, dC = host(g["dB"]), host(g["dC"])
    assert np.array_equal(dB[:, 0], DIM * rem), "dB state 0"
    assert np.array_equal(dC[:, 0], DIM * (pos + 1.0)), "dC state 0"
    assert not dB[:, 1:].any() and not dC[:, 1:].any(), "dB/dC of untouched states"
    dA = host(g["dA"])
    assert not dA[:, 1:].any()
    # dA sums rem*pos over every token: too large to be exact in fp32, so the fp32 bound applies
    want_dA0 = float(np.sum(np.where(pos != 0, rem * pos, 0.0)))
    assert np.all(np.abs(dA[:, 0] - want_dA0) <= 1e-4 * (1 + abs(want_dA0))), (dA[:4, 0], want_dA0)


@pytest.mark.parametrize("key,out_f32", [("0", True), ("1", True), ("2", True), ("3", True), ("4a", True),
                                         ("4a", False), ("4b", True)])
@pytest.mark.parametrize("width", [4, 3, 2])
def test_conv_probe(key, out_f32, width):
    import paper_2408_03865_amd as P
    cfg, pos = _pos(key)
    note(f"conv probe config {key} width {width} out_f32={out_f32}")
    Nb, L = cfg.batch, cfg.seqlen
    ones = np.ones((Nb, DIM, L), np.float32)
    w = np.broadcast_to(2.0 ** np.arange(width - 1, -1, -1), (DIM, width)).astype(np.float32)  # tap k -> 2^k
    x, dout = _act(ones, cfg.dtype), _act(ones, cfg.dtype)
    p = i32(pos)
    bias = f32(np.zeros(DIM))
    out = P.causal_conv1d_fwd(x, f32(w), bias, p, silu=False, out_f32=out_f32)
    dx, dw, db = P.causal_conv1d_bwd(x, f32(w), bias, p, dout, silu=False, out_f32=out_f32)
    torch().cuda.synchronize()
    taps = np.minimum(pos, width - 1) + 1
    want = (2.0 ** taps - 1)[:, None, :]
    assert np.array_equal(host(out), np.broadcast_to(want, (Nb, DIM, L)))
    wdx = np.zeros((Nb, L))
    for k in range(width):
        live = np.zeros((Nb, L), bool)
        live[:, :L - k] = pos[:, k:] >= k
        wdx += np.where(live, 2.0 ** k, 0.0)
    assert np.array_equal(host(dx), np.broadcast_to(wdx[:, None, :], (Nb, DIM, L))), "dx reverse mask"
    want_dw = np.array([np.count_nonzero(pos >= (width - 1 - j)) for j in range(width)], np.float64)
    assert np.array_equal(host(dw), np.broadcast_to(want_dw, (DIM, width)))
    assert np.array_equal(host(db), np.full(DIM, float(Nb * L)))
