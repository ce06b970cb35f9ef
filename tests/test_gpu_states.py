"""GPU parity for state passing across rows (a sequence cut at a row end continues in
another row, the future work of §5): the per-row initial and final states of both
operators and their gradients, against the oracle, and a row cut in two on the GPU
chained through the passed states against the uncut row."""
import numpy as np
import pytest

import workloads as W
from gpu_common import TOL, act, assert_close, f32, host, i32, note

pytestmark = pytest.mark.gpu


def _cfg(batch, dim, seqlen, dtype):
    return W.Config("states", "states", batch, seqlen, dim, 16, 4, dtype,
                    ("lognormal", 3.0, 1.0, 1, max(seqlen, 1)), 9100 + batch * 17 + dim * 3 + seqlen)


def _continued(d, offsets):
    """Rows whose first sequence continues one cut at the end of another row."""
    pos = d["pos"].copy()
    for b, off in enumerate(offsets):
        n = int(np.argmax(pos[b, 1:] == 0)) + 1 if np.any(pos[b, 1:] == 0) else pos.shape[1]
        pos[b, :n] += off
    d["pos"] = pos
    return d


def _state_inputs(d, dtype, seed):
    rng = np.random.default_rng(seed)
    Nb, Dn, _ = d["u"].shape
    N = d["A"].shape[1]
    rnd = (lambda a: W.bf16_round(a)) if dtype == "bf16" else (lambda a: a)
    return {
        "h0": rng.standard_normal((Nb, Dn, N)).astype(np.float32),
        "dhf": rng.standard_normal((Nb, Dn, N)).astype(np.float32),
        "xi": rnd(rng.standard_normal((Nb, Dn, 3)).astype(np.float32)),
        "dxf": rnd(rng.standard_normal((Nb, Dn, 3)).astype(np.float32)),
    }


def _gpu(d, s, dtype, out_f32):
    import torch
    import paper_2408_03865_amd as P
    g = {k: act(d[k], dtype) for k in W.ACTIVATIONS}
    for k in ("A", "D", "delta_bias", "w", "bias"):
        g[k] = f32(d[k])
    pos = i32(d["pos"])
    xi, dxf = act(s["xi"], dtype), act(s["dxf"], dtype)
    h0, dhf = f32(s["h0"]), f32(s["dhf"])
    r = {}
    r["conv_out"], r["xfinal"] = P.causal_conv1d_fwd(g["x"], g["w"], g["bias"], pos, out_f32=out_f32,
                                                     initial_x=xi, return_final=True)
    r["dx"], r["dw"], r["dbias"], r["dxinit"] = P.causal_conv1d_bwd(
        g["x"], g["w"], g["bias"], pos, g["dout"], out_f32=out_f32, initial_x=xi, dfinal_x=dxf)
    r["out"], st, r["hfinal"] = P.selective_scan_fwd(
        g["u"], g["delta"], g["A"], g["B"], g["C"], g["D"], g["z"], g["delta_bias"], True, pos,
        return_states=True, out_f32=out_f32, initial_state=h0, return_final=True)
    r.update(P.selective_scan_bwd(g["u"], g["delta"], g["A"], g["B"], g["C"], g["D"], g["z"],
                                  g["delta_bias"], True, pos, g["dout"], saved_states=st, out_f32=out_f32,
                                  initial_state=h0, dfinal_state=dhf))
    r2 = P.selective_scan_bwd(g["u"], g["delta"], g["A"], g["B"], g["C"], g["D"], g["z"],
                              g["delta_bias"], True, pos, g["dout"], out_f32=out_f32,
                              initial_state=h0, dfinal_state=dhf)
    torch.cuda.synchronize()
    r["_recomputed"] = r2
    return r


def _oracle(d, s):
    import oracle as O
    r = {}
    r["conv_out"], r["xfinal"] = O.conv1d_fwd(d["x"], d["w"], d["bias"], d["pos"], xinit=s["xi"],
                                              return_final=True)
    cg = O.conv1d_bwd(d["x"], d["w"], d["bias"], d["pos"], d["dout"], xinit=s["xi"], dxfinal=s["dxf"])
    r.update(dx=cg["dx"], dw=cg["dw"], dbias=cg["dbias"], dxinit=cg["dxinit"])
    args = dict(u=d["u"], delta=d["delta"], A=d["A"], B=d["B"], C=d["C"], D=d["D"], z=d["z"],
                delta_bias=d["delta_bias"], delta_softplus=True, pos=d["pos"])
    r["out"], r["hfinal"] = O.scan_fwd(**args, h0=s["h0"], return_final=True)
    r.update(O.scan_bwd(**args, dout=d["dout"], h0=s["h0"], dhfinal=s["dhf"]))
    r["dinitial_state"] = r.pop("dh0")
    return r


KEYS = ("conv_out", "dx", "dw", "dbias", "dxinit", "out", "hfinal", "du", "ddelta", "dz", "dA", "dB",
        "dC", "dD", "ddelta_bias", "dinitial_state")

# (batch, dim, seqlen): split rows (few blocks), unsplit rows (>= 768 blocks), ragged,
# rows shorter than the conv halo
SHAPES = [(2, 24, 1000), (3, 5, 2049), (48, 256, 600), (2, 8, 2), (1, 16, 300)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_states_match_oracle(shape, dtype):
    import paper_2408_03865_amd as P
    note(f"states {shape} {dtype} segments={P.segments(*shape)}")
    d = W.make_inputs(_cfg(*shape, dtype), variant="general")
    d = _continued(d, [37 + 5 * b if b % 2 == 0 else 0 for b in range(shape[0])])
    s = _state_inputs(d, dtype, seed=shape[1] + shape[2])
    r = _gpu(d, s, dtype, out_f32=(dtype == "bf16"))
    ref = _oracle(d, s)
    tol = TOL[dtype]
    for k in KEYS:
        assert_close(f"{shape} {dtype} {k}", host(r[k]), ref[k], tol)
    # the final inputs are copies: bit-exact
    assert np.array_equal(host(r["xfinal"]), ref["xfinal"]), "final_x must be an exact copy"
    # recomputing the states inside the backward gives the same bits
    for k in ("du", "ddelta", "dz", "dA", "dB", "dC", "dD", "ddelta_bias", "dinitial_state"):
        assert np.array_equal(host(r[k]), host(r["_recomputed"][k])), k


def test_cut_rows_chain_on_gpu():
    """A row cut at several points, each second part fed the first part's final states
    on the GPU: outputs and chained gradients equal the uncut row's (fp32)."""
    import torch
    import paper_2408_03865_amd as P
    cfg = _cfg(1, 32, 1500, "f32")
    d = W.make_inputs(cfg, variant="general")
    g = {k: f32(d[k]) for k in (*W.ACTIVATIONS, "A", "D", "delta_bias", "w", "bias")}
    pos = i32(d["pos"])
    sc = lambda u, dl, B, C, z, p, **kw: P.selective_scan_fwd(u, dl, g["A"], B, C, g["D"], z,
                                                             g["delta_bias"], True, p, **kw)
    sb = lambda u, dl, B, C, z, p, dout, **kw: P.selective_scan_bwd(u, dl, g["A"], B, C, g["D"], z,
                                                                   g["delta_bias"], True, p, dout, **kw)
    full_c = P.causal_conv1d_fwd(g["x"], g["w"], g["bias"], pos)
    full_cg = P.causal_conv1d_bwd(g["x"], g["w"], g["bias"], pos, g["dout"])
    full_y = sc(g["u"], g["delta"], g["B"], g["C"], g["z"], pos)
    full_g = sb(g["u"], g["delta"], g["B"], g["C"], g["z"], pos, g["dout"])
    for cut in (1, 100, 511, 512, 777, 1499):
        note(f"cut at {cut}")
        a = {k: v[..., :cut].clone() for k, v in g.items() if k in W.ACTIVATIONS}
        b = {k: v[..., cut:].clone() for k, v in g.items() if k in W.ACTIVATIONS}
        pa, pb = pos[:, :cut].clone(), pos[:, cut:].clone()      # fresh, 16-byte aligned
        c1, xf = P.causal_conv1d_fwd(a["x"], g["w"], g["bias"], pa, return_final=True)
        c2 = P.causal_conv1d_fwd(b["x"], g["w"], g["bias"], pb, initial_x=xf)
        dx2, dw2, db2, dxi2 = P.causal_conv1d_bwd(b["x"], g["w"], g["bias"], pb, b["dout"], initial_x=xf)
        dx1, dw1, db1 = P.causal_conv1d_bwd(a["x"], g["w"], g["bias"], pa, a["dout"], dfinal_x=dxi2)
        y1, hf = sc(a["u"], a["delta"], a["B"], a["C"], a["z"], pa, return_final=True)
        y2 = sc(b["u"], b["delta"], b["B"], b["C"], b["z"], pb, initial_state=hf)
        g2 = sb(b["u"], b["delta"], b["B"], b["C"], b["z"], pb, b["dout"], initial_state=hf)
        g1 = sb(a["u"], a["delta"], a["B"], a["C"], a["z"], pa, a["dout"], dfinal_state=g2["dinitial_state"])
        torch.cuda.synchronize()
        tol = TOL["f32"]
        assert_close(f"cut {cut} conv", host(torch.cat([c1, c2], -1)), host(full_c), tol)
        assert_close(f"cut {cut} dx", host(torch.cat([dx1, dx2], -1)), host(full_cg[0]), tol)
        assert_close(f"cut {cut} dw", host(dw1 + dw2), host(full_cg[1]), tol)
        assert_close(f"cut {cut} dbias", host(db1 + db2), host(full_cg[2]), tol)
        assert_close(f"cut {cut} y", host(torch.cat([y1, y2], -1)), host(full_y), tol)
        for k in ("du", "ddelta", "dz", "dB", "dC"):
            assert_close(f"cut {cut} {k}", host(torch.cat([g1[k], g2[k]], -1)), host(full_g[k]), tol)
        for k in ("dA", "dD", "ddelta_bias"):
            assert_close(f"cut {cut} {k}", host(g1[k] + g2[k]), host(full_g[k]), tol)


def test_check_position_indices_continued():
    import paper_2408_03865_amd as P
    pos = W.positions_from_lengths([[3, 5], [8]], 8)
    pos[0, :3] = [4, 5, 6]
    t = i32(pos)
    assert not P.check_position_indices(t)
    assert P.check_position_indices(t, continued=True)
    pos[1, 0] = -2
    assert not P.check_position_indices(i32(pos), continued=True)


def test_cut_plan_rows_chained_on_gpu():
    """A stream packed by the cut policy (rows filled to the end, sequences continued in
    the next row), the rows run one after another on the GPU with the previous row's
    final states: every output against the same chain on the oracle (fp32)."""
    import torch
    import oracle as O
    import paper_2408_03865_amd as P
    L, Dn = 1024, 32
    ln = W.draw_stream_lengths(("lognormal", 6.0, 1.0, 16, 4096), np.random.default_rng(11), 12)
    pieces, rows = P.pack_plan(ln, L, "cut")
    pos = P.pack_positions(pieces, rows, L)
    d = W.make_inputs(_cfg(rows, Dn, L, "f32"), variant="general")
    d["pos"] = pos
    g = {k: f32(d[k]) for k in (*W.ACTIVATIONS, "A", "D", "delta_bias", "w", "bias")}
    sargs = lambda t, p: (t["u"], t["delta"], t["A"], t["B"], t["C"], t["D"], t["z"], t["delta_bias"], True, p)
    xi = hi = None
    oxi = ohi = None
    for r in range(rows):
        note(f"cut-plan row {r}")
        t = {k: (v[r:r + 1].clone() if k in W.ACTIVATIONS else v) for k, v in g.items()}
        p = i32(pos[r:r + 1])
        c, xf = P.causal_conv1d_fwd(t["x"], t["w"], t["bias"], p, initial_x=xi, return_final=True)
        y, hf = P.selective_scan_fwd(*sargs(t, p), initial_state=hi, return_final=True)
        torch.cuda.synchronize()
        od = {k: d[k][r:r + 1] for k in W.ACTIVATIONS}
        oc, oxf = O.conv1d_fwd(od["x"], d["w"], d["bias"], pos[r:r + 1], xinit=oxi, return_final=True)
        oy, ohf = O.scan_fwd(od["u"], od["delta"], d["A"], od["B"], od["C"], d["D"], od["z"], d["delta_bias"],
                             True, pos[r:r + 1], h0=ohi, return_final=True)
        assert_close(f"row {r} conv", host(c), oc, TOL["f32"])
        assert_close(f"row {r} y", host(y), oy, TOL["f32"])
        assert_close(f"row {r} final state", host(hf), ohf, TOL["f32"])
        assert np.array_equal(host(xf), oxf)
        xi, hi, oxi, ohi = xf, hf, oxf, ohf
