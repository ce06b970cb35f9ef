"""Host packing plans (§3.1, §5) from the library's C++ planner: structure of the plans,
their position indices, padding rates, and end to end through the oracle: packed rows
(with state passing between the rows of the cut policy) reproduce the per-sequence runs."""
import numpy as np
import pytest

import oracle as O
import workloads as W


def _P():
    import paper_2408_03865_amd as P
    return P


def _stream(seed=0, n=400, hi=300):
    rng = np.random.default_rng(seed)
    ln = W.draw_stream_lengths(("lognormal", 4.0, 1.0, 1, hi), rng, n)
    return ln


@pytest.mark.parametrize("policy", ["sequential", "greedy", "cut"])
def test_plan_structure(policy):
    P = _P()
    L = 256
    ln = _stream(1)
    ln[5] = 700                      # longer than a row
    pieces, rows = P.pack_plan(ln, L, policy, window=32)
    seq, row, off, length, first = pieces.T
    assert np.all(length > 0) and np.all(off >= 0) and np.all(off + length <= L)
    assert np.all((row >= 0) & (row < rows))
    # pieces of a row do not overlap
    for r in range(rows):
        sel = np.flatnonzero(row == r)
        o = np.sort(off[sel])
        e = (off[sel] + length[sel])[np.argsort(off[sel])]
        assert np.all(o[1:] >= e[:-1])
    # every sequence is placed, its pieces consecutive in position
    for i, n in enumerate(ln):
        sel = np.flatnonzero(seq == i)
        assert sel.size >= 1
        f = first[sel]
        assert f[0] == 0 and np.all(f[1:] == (f + length[sel])[:-1])
        total = length[sel].sum()
        assert total == (n if policy == "cut" else min(n, L))
    if policy == "sequential":
        # received order, row by row
        key = row * L + off
        assert np.all(np.diff(key) > 0)
    if policy == "cut":
        # only the last row holds padding; a piece continuing a sequence starts a row
        fill = np.bincount(row, weights=length, minlength=rows)
        assert np.all(fill[:-1] == L)
        assert np.all(off[first > 0] == 0)
    else:
        assert np.all(first == 0)


def test_positions_and_contract():
    P = _P()
    L = 200
    ln = _stream(2, n=120)
    for policy in ("sequential", "greedy", "cut"):
        pieces, rows = P.pack_plan(ln, L, policy, window=16)
        pos = P.pack_positions(pieces, rows, L)
        assert pos.shape == (rows, L)
        assert O.check_positions(pos, continued=(policy == "cut")) == -1, policy
        for s, r, o, n, f in pieces[:50]:
            assert np.array_equal(pos[r, o:o + n], np.arange(f, f + n)), (policy, s)


def test_padding_rates_order():
    """On the synthetic Mamba-1.4B length law (mean ≈ 646 tokens, rows of 4096):
    greedy with a large window pads less than sequential, and cutting pads only the
    last row."""
    P = _P()
    ln = W.draw_stream_lengths(("lognormal", 6.0, 1.0, 16, 4096), np.random.default_rng(3), 5000)
    rate = {}
    for policy, w in (("sequential", 1), ("greedy", 1024), ("cut", 1)):
        pieces, rows = P.pack_plan(ln, 4096, policy, window=w)
        rate[policy] = P.padding_rate(pieces, rows, 4096)
    assert 0.08 < rate["sequential"] < 0.25
    assert rate["greedy"] < 0.02
    assert rate["cut"] < 4096 / (ln.sum())
    assert rate["cut"] <= rate["greedy"] <= rate["sequential"]


def test_errors():
    import ctypes
    from paper_2408_03865_amd import _lib
    P = _P()
    lib = _lib.load()
    n1, n2 = ctypes.c_int64(), ctypes.c_int64()
    ln = np.array([3, 0, 4], dtype=np.int64)
    assert lib.packmamba_pack_plan(ln.ctypes.data, 3, 8, 0, 1, None, 0, ctypes.byref(n1), ctypes.byref(n2)) == 2
    ln = np.array([3, 5, 4], dtype=np.int64)
    assert lib.packmamba_pack_plan(ln.ctypes.data, 3, 8, 9, 1, None, 0, ctypes.byref(n1), ctypes.byref(n2)) == 3
    assert lib.packmamba_pack_plan(ln.ctypes.data, 3, 8, 1, 0, None, 0, ctypes.byref(n1), ctypes.byref(n2)) == 2
    out = np.zeros((1, 5), dtype=np.int64)
    assert lib.packmamba_pack_plan(ln.ctypes.data, 3, 8, 0, 1, out.ctypes.data, 1, ctypes.byref(n1),
                                   ctypes.byref(n2)) == 5
    assert n1.value == 3 and n2.value == 2
    with pytest.raises(_lib.PackMambaError):
        P.pack_positions(np.array([[0, 0, 5, 4, 0]]), 1, 8)          # piece past the row end


def _sequences_data(ln, Dn, N, W_, seed):
    rng = np.random.default_rng(seed)
    seqs = []
    for n in ln:
        seqs.append({k: rng.standard_normal((Dn, n)) for k in ("x", "u", "delta", "z", "dout")}
                    | {k: rng.standard_normal((N, n)) for k in ("B", "C")})
    par = dict(A=-np.exp(rng.normal(0, 0.5, (Dn, N))), D=rng.standard_normal(Dn),
               delta_bias=rng.uniform(-1, 0.5, Dn), w=rng.uniform(-0.5, 0.5, (Dn, W_)),
               bias=rng.uniform(-0.5, 0.5, Dn))
    return seqs, par


def _scatter(pieces, rows, L, seqs, Dn, N):
    act = {k: np.zeros((rows, Dn, L)) for k in ("x", "u", "delta", "z", "dout")}
    bc = {k: np.zeros((rows, N, L)) for k in ("B", "C")}
    for s, r, o, n, f in pieces:
        for k in act:
            act[k][r, :, o:o + n] = seqs[s][k][:, f:f + n]
        for k in bc:
            bc[k][r, :, o:o + n] = seqs[s][k][:, f:f + n]
    return act | bc


@pytest.mark.parametrize("policy", ["sequential", "greedy", "cut"])
def test_packed_rows_reproduce_sequences(policy):
    """Packing by the plan changes nothing (PUI, §3.1); for the cut policy the rows are run
    in order, each taking the previous row's final states, and the gradients run back
    through the state gradients."""
    P = _P()
    Dn, N, W_, L = 2, 3, 4, 48
    ln = np.array([30, 5, 70, 1, 2, 40, 17, 9, 60, 3], dtype=np.int64)
    if policy != "cut":
        ln = np.minimum(ln, L)
    seqs, par = _sequences_data(ln, Dn, N, W_, seed=5)
    pieces, rows = P.pack_plan(ln, L, policy, window=4)
    pos = P.pack_positions(pieces, rows, L)
    t = _scatter(pieces, rows, L, seqs, Dn, N)
    sargs = lambda tt, p: dict(u=tt["u"], delta=tt["delta"], A=par["A"], B=tt["B"], C=tt["C"], D=par["D"],
                               z=tt["z"], delta_bias=par["delta_bias"], delta_softplus=True, pos=p)
    # packed rows, chained through the states row by row
    conv_out = np.zeros((rows, Dn, L)); y = np.zeros((rows, Dn, L))
    xi = hi = None
    for r in range(rows):
        sl = slice(r, r + 1)
        tr = {k: v[sl] for k, v in t.items()}
        c, xi = O.conv1d_fwd(tr["x"], par["w"], par["bias"], pos[sl], xinit=xi, return_final=True)
        o, hi = O.scan_fwd(**sargs(tr, pos[sl]), h0=hi, return_final=True)
        conv_out[r], y[r] = c[0], o[0]
    # backward, last row first
    du = np.zeros((rows, Dn, L)); dx = np.zeros((rows, Dn, L))
    dA = 0.0; dw = 0.0
    dhf = dxf = None
    for r in reversed(range(rows)):
        sl = slice(r, r + 1)
        tr = {k: v[sl] for k, v in t.items()}
        # initial states of this row: the previous row's final states (forward again)
        h0 = x0 = None
        if r > 0:
            h0 = np.zeros((1, Dn, N)); x0 = np.zeros((1, Dn, W_ - 1))
            for q in range(r):
                tq = {k: v[q:q + 1] for k, v in t.items()}
                _, x0 = O.conv1d_fwd(tq["x"], par["w"], par["bias"], pos[q:q + 1], xinit=x0 if q else None,
                                     return_final=True)
                _, h0 = O.scan_fwd(**sargs(tq, pos[q:q + 1]), h0=h0 if q else None, return_final=True)
        g = O.scan_bwd(**sargs(tr, pos[sl]), dout=tr["dout"], h0=h0, dhfinal=dhf)
        cg = O.conv1d_bwd(tr["x"], par["w"], par["bias"], pos[sl], tr["dout"], xinit=x0, dxfinal=dxf)
        du[r], dx[r] = g["du"][0], cg["dx"][0]
        dA, dw = dA + g["dA"], dw + cg["dw"]
        dhf, dxf = g["dh0"], cg["dxinit"]
    # per-sequence references
    rdA = 0.0; rdw = 0.0
    for s, n in enumerate(ln):
        one = {k: v[None] for k, v in seqs[s].items()}
        p1 = np.arange(n, dtype=np.int32)[None]
        c_ref = O.conv1d_fwd(one["x"], par["w"], par["bias"], p1)
        y_ref = O.scan_fwd(**sargs(one, p1))
        g_ref = O.scan_bwd(**sargs(one, p1), dout=one["dout"])
        cg_ref = O.conv1d_bwd(one["x"], par["w"], par["bias"], p1, one["dout"])
        rdA, rdw = rdA + g_ref["dA"], rdw + cg_ref["dw"]
        for _, r, o, m, f in pieces[pieces[:, 0] == s]:
            np.testing.assert_allclose(conv_out[r, :, o:o + m], c_ref[0, :, f:f + m], rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(y[r, :, o:o + m], y_ref[0, :, f:f + m], rtol=1e-11, atol=1e-11)
            np.testing.assert_allclose(du[r, :, o:o + m], g_ref["du"][0, :, f:f + m], rtol=1e-10, atol=1e-10)
            np.testing.assert_allclose(dx[r, :, o:o + m], cg_ref["dx"][0, :, f:f + m], rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dA, rdA, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(dw, rdw, rtol=1e-11, atol=1e-11)
