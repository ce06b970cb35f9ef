"""Pins for the fp64 oracle: checks against facts that do not come from the oracle.

Each pin takes an oracle library handle (so the same pins can be run against
deliberately broken builds of the oracle) and raises AssertionError on failure.

  pin_pui_*           packed result == per-sequence unpacked results (§3.1, PUI)
  pin_closed_scan     constant step, B and u inside a sequence: the geometric sum
                      that Eq. (3) reduces to
  pin_closed_conv     constant x inside a sequence: the sum of the live taps
  pin_fd_*            central finite differences of every gradient
  pin_len1_*          every sequence has length 1 (every token resets)
  pin_cumsum          N=1, A=0, unit step, B=C=1: the per-sequence prefix sum
  pin_library_conv    torch's conv1d (fp64, CPU) run per sequence
  pin_states          chunk-end hidden states against the geometric sum
  pin_check_positions the index contract of §3.1
  pin_split_*         a row cut in two, the parts passing states (§5): equal to the
                      uncut row, forward and backward (gradients chained through
                      the passed states)
  pin_fd_*_states     finite differences of the initial-state gradients, on rows
                      that continue a sequence
"""
from __future__ import annotations

import numpy as np

import oracle as O
import workloads as W


def _close(a, b, rtol, what):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, (what, a.shape, b.shape)
    err = np.abs(a - b) / (1.0 + np.abs(b))
    m = float(err.max()) if err.size else 0.0
    assert m <= rtol, f"{what}: max scaled error {m:.3e} > {rtol:.1e}"


def _sigmoid(v):
    return 1.0 / (1.0 + np.exp(-v))


def _softplus(s):
    return np.where(s > 20.0, s, np.log1p(np.exp(np.minimum(s, 20.0))))


def _problem(rows, Dn=3, N=4, Wd=4, seed=0, general=True):
    """Small random problem with the given per-row sequence lengths."""
    rng = np.random.default_rng(seed)
    Nb, L = len(rows), sum(rows[0])
    p = dict(
        x=rng.standard_normal((Nb, Dn, L)), u=rng.standard_normal((Nb, Dn, L)),
        delta=rng.standard_normal((Nb, Dn, L)), z=rng.standard_normal((Nb, Dn, L)),
        B=rng.standard_normal((Nb, N, L)), C=rng.standard_normal((Nb, N, L)),
        A=-np.exp(rng.normal(0, 0.5, (Dn, N))), D=rng.standard_normal(Dn),
        delta_bias=rng.uniform(-1, 0.5, Dn), w=rng.uniform(-0.5, 0.5, (Dn, Wd)),
        bias=rng.uniform(-0.5, 0.5, Dn), dout=rng.standard_normal((Nb, Dn, L)),
        pos=W.positions_from_lengths(rows, L), rows=rows,
    )
    if not general:
        p["A"] = -np.broadcast_to(np.arange(1, N + 1, dtype=np.float64), (Dn, N)).copy()
    return p


def _scan_args(p, **kw):
    a = dict(u=p["u"], delta=p["delta"], A=p["A"], B=p["B"], C=p["C"], D=p["D"], z=p["z"],
             delta_bias=p["delta_bias"], delta_softplus=True, pos=p["pos"])
    a.update(kw)
    return a


# ---------------------------------------------------------------------------
# (a) packing-unpacking invariance
# ---------------------------------------------------------------------------

PUI_ROWS = [[7, 1, 12, 1, 1, 18], [40]]


def _sequences(p):
    """Split a packed problem into its sequences: list of (row, start, length)."""
    out = []
    for b, row in enumerate(p["rows"]):
        s = 0
        for n in row:
            out.append((b, s, n))
            s += n
    return out


def pin_pui_scan(lib):
    p = _problem(PUI_ROWS, seed=1)
    packed_out = O.scan_fwd(**_scan_args(p), lib=lib)
    packed_g = O.scan_bwd(**_scan_args(p), dout=p["dout"], lib=lib)
    acc = {k: 0.0 for k in ("dA", "dD", "ddelta_bias")}
    for b, s, n in _sequences(p):
        sl = slice(s, s + n)
        one = {k: p[k][b:b + 1, :, sl] for k in ("u", "delta", "z", "B", "C", "dout")}
        q = dict(p, **one, pos=np.arange(n, dtype=np.int32)[None])
        out = O.scan_fwd(**_scan_args(q), lib=lib)
        g = O.scan_bwd(**_scan_args(q), dout=q["dout"], lib=lib)
        _close(packed_out[b:b + 1, :, sl], out, 1e-12, "PUI scan out")
        for k in ("du", "ddelta", "dz", "dB", "dC"):
            _close(packed_g[k][b:b + 1, :, sl], g[k], 1e-12, f"PUI scan {k}")
        for k in acc:
            acc[k] = acc[k] + g[k]
    for k in acc:
        _close(packed_g[k], acc[k], 1e-12, f"PUI scan {k} (sum over sequences)")


def pin_pui_conv(lib):
    p = _problem(PUI_ROWS, seed=2)
    out = O.conv1d_fwd(p["x"], p["w"], p["bias"], p["pos"], silu=True, lib=lib)
    g = O.conv1d_bwd(p["x"], p["w"], p["bias"], p["pos"], p["dout"], silu=True, lib=lib)
    dw, db = 0.0, 0.0
    for b, s, n in _sequences(p):
        sl = slice(s, s + n)
        pos = np.arange(n, dtype=np.int32)[None]
        o1 = O.conv1d_fwd(p["x"][b:b + 1, :, sl], p["w"], p["bias"], pos, silu=True, lib=lib)
        g1 = O.conv1d_bwd(p["x"][b:b + 1, :, sl], p["w"], p["bias"], pos, p["dout"][b:b + 1, :, sl],
                          silu=True, lib=lib)
        _close(out[b:b + 1, :, sl], o1, 1e-12, "PUI conv out")
        _close(g["dx"][b:b + 1, :, sl], g1["dx"], 1e-12, "PUI conv dx")
        dw, db = dw + g1["dw"], db + g1["dbias"]
    _close(g["dw"], dw, 1e-12, "PUI conv dw")
    _close(g["dbias"], db, 1e-12, "PUI conv dbias")


# ---------------------------------------------------------------------------
# (b) closed forms
# ---------------------------------------------------------------------------

def pin_closed_scan(lib):
    """Constant step dt, B_n and u inside each sequence.

    With a_n = exp(dt A_n) and beta_n = dt B_n u, the state after the token with
    position index t is beta_n (1 - a_n^(t+1)) / (1 - a_n): the geometric sum that
    Eq. (3) gives when every term is equal.
    """
    rows = [[9, 1, 30], [25, 15]]
    p = _problem(rows, Dn=2, N=5, seed=3)
    Nb, Dn, L = p["u"].shape
    N = p["A"].shape[1]
    for b, s, n in _sequences(p):
        sl = slice(s, s + n)
        p["u"][b, :, sl] = p["u"][b, :, s:s + 1]
        p["delta"][b, :, sl] = p["delta"][b, :, s:s + 1]
        p["B"][b, :, sl] = p["B"][b, :, s:s + 1]
    out = O.scan_fwd(**_scan_args(p), lib=lib)
    dt = _softplus(p["delta"] + p["delta_bias"][None, :, None])              # (Nb, Dn, L)
    t = p["pos"][:, None, None, :].astype(np.float64)                       # (Nb,1,1,L)
    a = np.exp(dt[:, :, None, :] * p["A"][None, :, :, None])                # (Nb,Dn,N,L)
    beta = dt[:, :, None, :] * p["B"][:, None, :, :] * p["u"][:, :, None, :]
    h = beta * (1.0 - a ** (t + 1.0)) / (1.0 - a)
    y = np.einsum("bnl,bdnl->bdl", p["C"], h)
    ref = (y + p["D"][None, :, None] * p["u"]) * p["z"] * _sigmoid(p["z"])
    _close(out, ref, 1e-12, "closed-form scan")


def pin_states(lib):
    rows = [[50, 14, 64, 1, 63], [192]]
    p = _problem(rows, Dn=2, N=3, seed=4)
    for b, s, n in _sequences(p):
        sl = slice(s, s + n)
        for k in ("u", "delta"):
            p[k][b, :, sl] = p[k][b, :, s:s + 1]
        p["B"][b, :, sl] = p["B"][b, :, s:s + 1]
    stride = 64
    st = O.scan_states(p["u"], p["delta"], p["A"], p["B"], p["delta_bias"], True, p["pos"], stride,
                       lib=lib)
    dt = _softplus(p["delta"] + p["delta_bias"][None, :, None])
    L = p["u"].shape[2]
    for c in range((L + stride - 1) // stride):
        l = min((c + 1) * stride, L) - 1
        tt = p["pos"][:, l].astype(np.float64)[:, None, None]
        a = np.exp(dt[:, :, l][:, :, None] * p["A"][None])
        beta = dt[:, :, l][:, :, None] * p["B"][:, None, :, l] * p["u"][:, :, l][:, :, None]
        _close(st[:, :, c, :], beta * (1 - a ** (tt + 1)) / (1 - a), 1e-12, f"states chunk {c}")


def pin_closed_conv(lib):
    """Constant x = c inside a sequence: pre-activation = bias + c * (sum of live taps)."""
    rows = [[1, 2, 3, 10, 4], [20]]
    p = _problem(rows, Dn=3, seed=5)
    Wd = p["w"].shape[1]
    for b, s, n in _sequences(p):
        p["x"][b, :, s:s + n] = p["x"][b, :, s:s + 1]
    out = O.conv1d_fwd(p["x"], p["w"], p["bias"], p["pos"], silu=False, lib=lib)
    ref = np.empty_like(out)
    for b in range(out.shape[0]):
        for l in range(out.shape[2]):
            kmax = min(Wd - 1, int(p["pos"][b, l]))
            taps = p["w"][:, Wd - 1 - kmax:].sum(axis=1)
            ref[b, :, l] = p["bias"] + p["x"][b, :, l] * taps
    _close(out, ref, 1e-13, "closed-form conv")
    out2 = O.conv1d_fwd(p["x"], p["w"], p["bias"], p["pos"], silu=True, lib=lib)
    _close(out2, ref * _sigmoid(ref), 1e-13, "closed-form conv + SiLU")


# ---------------------------------------------------------------------------
# (c) central finite differences
# ---------------------------------------------------------------------------

FD_ROWS = [[4, 1, 7], [12]]


def _fd(fun, params, names, grads, what, rtol=1e-7):
    for k in names:
        arr = params[k]
        num = np.zeros_like(arr)
        it = np.nditer(arr, flags=["multi_index"])
        for _ in it:
            i = it.multi_index
            v = arr[i]
            eps = 1e-6 * max(1.0, abs(v))
            arr[i] = v + eps
            fp = fun()
            arr[i] = v - eps
            fm = fun()
            arr[i] = v
            num[i] = (fp - fm) / (2 * eps)
        _close(grads[k], num, rtol, f"{what} d{k} vs finite differences")


def pin_fd_scan(lib):
    p = _problem(FD_ROWS, Dn=2, N=3, seed=6)

    def loss():
        return float(np.sum(p["dout"] * O.scan_fwd(**_scan_args(p), lib=lib)))

    g = O.scan_bwd(**_scan_args(p), dout=p["dout"], lib=lib)
    grads = {"u": g["du"], "delta": g["ddelta"], "A": g["dA"], "B": g["dB"], "C": g["dC"],
             "D": g["dD"], "z": g["dz"], "delta_bias": g["ddelta_bias"]}
    _fd(loss, p, list(grads), grads, "scan")


def pin_fd_scan_plain(lib):
    """No D, no z, no delta_bias, no softplus: the bare recurrence and its gradients."""
    p = _problem(FD_ROWS, Dn=2, N=3, seed=7)
    kw = dict(D=None, z=None, delta_bias=None, delta_softplus=False)
    p["delta"] = np.abs(p["delta"]) * 0.5 + 0.1

    def loss():
        return float(np.sum(p["dout"] * O.scan_fwd(**_scan_args(p, **kw), lib=lib)))

    g = O.scan_bwd(**_scan_args(p, **kw), dout=p["dout"], lib=lib)
    grads = {"u": g["du"], "delta": g["ddelta"], "A": g["dA"], "B": g["dB"], "C": g["dC"]}
    _fd(loss, p, list(grads), grads, "scan (plain)")


def pin_fd_conv(lib):
    for silu in (True, False):
        p = _problem(FD_ROWS, Dn=2, seed=8 + silu)

        def loss():
            return float(np.sum(p["dout"] * O.conv1d_fwd(p["x"], p["w"], p["bias"], p["pos"], silu,
                                                          lib=lib)))

        g = O.conv1d_bwd(p["x"], p["w"], p["bias"], p["pos"], p["dout"], silu, lib=lib)
        _fd(loss, p, ["x", "w", "bias"], {"x": g["dx"], "w": g["dw"], "bias": g["dbias"]},
            f"conv silu={silu}")


# ---------------------------------------------------------------------------
# special cases
# ---------------------------------------------------------------------------

def pin_len1_scan(lib):
    """Every token starts a sequence: out = (dt u sum_n C_n B_n + D u) SiLU(z)."""
    p = _problem([[1] * 16], Dn=3, N=4, seed=10)
    out = O.scan_fwd(**_scan_args(p), lib=lib)
    dt = _softplus(p["delta"] + p["delta_bias"][None, :, None])
    cb = np.sum(p["C"] * p["B"], axis=1)[:, None, :]
    ref = (dt * p["u"] * cb + p["D"][None, :, None] * p["u"]) * p["z"] * _sigmoid(p["z"])
    _close(out, ref, 1e-13, "all-length-1 scan")
    g = O.scan_bwd(**_scan_args(p), dout=p["dout"], lib=lib)
    assert np.all(g["dA"] == 0.0), "dA must vanish when every multiplier is a reset"


def pin_len1_conv(lib):
    p = _problem([[1] * 16], Dn=3, seed=11)
    out = O.conv1d_fwd(p["x"], p["w"], p["bias"], p["pos"], silu=False, lib=lib)
    _close(out, p["bias"][None, :, None] + p["w"][None, :, -1:] * p["x"], 1e-14, "all-length-1 conv")


def pin_cumsum(lib):
    """N=1, A=0, delta=1 without softplus, B=C=1: y is the prefix sum of u per sequence."""
    rows = [[5, 1, 1, 9, 24], [40]]
    p = _problem(rows, Dn=2, N=1, seed=12)
    Nb, Dn, L = p["u"].shape
    out = O.scan_fwd(p["u"], np.ones_like(p["u"]), np.zeros((Dn, 1)), np.ones((Nb, 1, L)),
                     np.ones((Nb, 1, L)), None, None, None, False, p["pos"], lib=lib)
    ref = np.empty_like(out)
    for b, s, n in _sequences(p):
        ref[b, :, s:s + n] = np.cumsum(p["u"][b, :, s:s + n], axis=-1)
    _close(out, ref, 1e-14, "segmented cumsum")


def pin_library_conv(lib):
    """torch.nn.functional.conv1d (fp64, CPU) applied to each sequence separately."""
    import torch
    import torch.nn.functional as F
    rows = [[3, 1, 17, 2, 9], [32]]
    p = _problem(rows, Dn=4, seed=13)
    out = O.conv1d_fwd(p["x"], p["w"], p["bias"], p["pos"], silu=True, lib=lib)
    Wd = p["w"].shape[1]
    w = torch.from_numpy(p["w"])[:, None, :]
    bias = torch.from_numpy(p["bias"])
    for b, s, n in _sequences(p):
        xs = torch.from_numpy(np.ascontiguousarray(p["x"][b:b + 1, :, s:s + n]))
        ref = F.silu(F.conv1d(xs, w, bias, padding=Wd - 1, groups=xs.shape[1])[..., :n])
        _close(out[b:b + 1, :, s:s + n], ref.numpy(), 1e-14, "library conv")


def pin_check_positions(lib):
    good = W.positions_from_lengths([[3, 1, 4], [8]], 8)
    assert O.check_positions(good, lib=lib) == -1
    bad = good.copy(); bad[0, 0] = 1
    assert O.check_positions(bad, lib=lib) == 0
    bad = good.copy(); bad[1, 5] = 7
    assert O.check_positions(bad, lib=lib) == 8 + 5
    bad = good.copy(); bad[0, 2] = 0; bad[0, 3] = 2
    assert O.check_positions(bad, lib=lib) == 3


# ---------------------------------------------------------------------------
# state passing across rows (§5): cutting a row and passing the states must not
# change anything
# ---------------------------------------------------------------------------

SPLIT_ROWS = [[6, 1, 9, 2, 14], [32]]
# cut points: inside a sequence, on a sequence start, just before a start, a part
# shorter than the conv halo, inside the single long sequence
SPLIT_CUTS = [(0, 3), (0, 6), (0, 15), (0, 30), (1, 1), (1, 17)]


def _cut(p, b, c, keys):
    first = {k: p[k][b:b + 1, ..., :c] for k in keys}
    second = {k: p[k][b:b + 1, ..., c:] for k in keys}
    return first, second


def pin_split_scan(lib):
    p = _problem(SPLIT_ROWS, Dn=2, N=3, seed=20)
    full_out = O.scan_fwd(**_scan_args(p), lib=lib)
    full_g = O.scan_bwd(**_scan_args(p), dout=p["dout"], lib=lib)
    keys = ("u", "delta", "z", "B", "C", "dout", "pos")
    for b, c in SPLIT_CUTS:
        one, two = _cut(p, b, c, keys)
        q1, q2 = dict(p, **one), dict(p, **two)
        o1, h1 = O.scan_fwd(**_scan_args(q1), lib=lib, return_final=True)
        o2, h2 = O.scan_fwd(**_scan_args(q2), lib=lib, h0=h1, return_final=True)
        _close(np.concatenate([o1, o2], axis=-1), full_out[b:b + 1], 1e-12, f"split scan out {b},{c}")
        _, hfull = O.scan_fwd(**_scan_args(dict(p, **{k: p[k][b:b + 1] for k in keys})), lib=lib,
                              return_final=True)
        _close(h2, hfull, 1e-12, f"split scan final state {b},{c}")
        g2 = O.scan_bwd(**_scan_args(q2), dout=q2["dout"], lib=lib, h0=h1)
        g1 = O.scan_bwd(**_scan_args(q1), dout=q1["dout"], lib=lib, dhfinal=g2["dh0"])
        for k in ("du", "ddelta", "dz", "dB", "dC"):
            _close(np.concatenate([g1[k], g2[k]], axis=-1), full_g[k][b:b + 1], 1e-11,
                   f"split scan {k} {b},{c}")
        one_row = dict(p, **{k: p[k][b:b + 1] for k in keys})
        gr = O.scan_bwd(**_scan_args(one_row), dout=one_row["dout"], lib=lib)
        for k in ("dA", "dD", "ddelta_bias"):
            _close(g1[k] + g2[k], gr[k], 1e-11, f"split scan {k} {b},{c}")
        if p["pos"][b, c] == 0:
            assert np.all(g2["dh0"] == 0.0), "a start at the cut must stop the state's gradient"


def pin_split_conv(lib):
    p = _problem(SPLIT_ROWS, Dn=2, seed=21)
    for silu in (True, False):
        full = O.conv1d_fwd(p["x"], p["w"], p["bias"], p["pos"], silu, lib=lib)
        for b, c in SPLIT_CUTS:
            one, two = _cut(p, b, c, ("x", "dout", "pos"))
            o1, f1 = O.conv1d_fwd(one["x"], p["w"], p["bias"], one["pos"], silu, lib=lib, return_final=True)
            o2 = O.conv1d_fwd(two["x"], p["w"], p["bias"], two["pos"], silu, lib=lib, xinit=f1)
            _close(np.concatenate([o1, o2], axis=-1), full[b:b + 1], 1e-13, f"split conv out {b},{c}")
            gfull = O.conv1d_bwd(p["x"][b:b + 1], p["w"], p["bias"], p["pos"][b:b + 1],
                                 p["dout"][b:b + 1], silu, lib=lib)
            g2 = O.conv1d_bwd(two["x"], p["w"], p["bias"], two["pos"], two["dout"], silu, lib=lib, xinit=f1)
            g1 = O.conv1d_bwd(one["x"], p["w"], p["bias"], one["pos"], one["dout"], silu, lib=lib,
                              dxfinal=g2["dxinit"])
            _close(np.concatenate([g1["dx"], g2["dx"]], axis=-1), gfull["dx"], 1e-12, f"split conv dx {b},{c}")
            _close(g1["dw"] + g2["dw"], gfull["dw"], 1e-12, f"split conv dw {b},{c}")
            _close(g1["dbias"] + g2["dbias"], gfull["dbias"], 1e-12, f"split conv dbias {b},{c}")


def pin_fd_scan_states(lib):
    """A row continuing a sequence (first index 5) from an initial state, with a final-state
    gradient: finite differences of every input, the initial state included."""
    p = _problem([[3, 9]], Dn=2, N=3, seed=22)
    p["pos"][0, :3] = np.arange(5, 8)
    rng = np.random.default_rng(23)
    p["h0"] = rng.standard_normal((1, 2, 3))
    ghf = rng.standard_normal((1, 2, 3))

    def loss():
        out, hf = O.scan_fwd(**_scan_args(p), lib=lib, h0=p["h0"], return_final=True)
        return float(np.sum(p["dout"] * out) + np.sum(ghf * hf))

    g = O.scan_bwd(**_scan_args(p), dout=p["dout"], lib=lib, h0=p["h0"], dhfinal=ghf)
    grads = {"u": g["du"], "delta": g["ddelta"], "A": g["dA"], "B": g["dB"], "C": g["dC"],
             "D": g["dD"], "z": g["dz"], "delta_bias": g["ddelta_bias"], "h0": g["dh0"]}
    _fd(loss, p, list(grads), grads, "scan with states")


def pin_fd_conv_states(lib):
    for silu in (True, False):
        p = _problem([[2, 1, 6]], Dn=2, seed=24 + silu)
        p["pos"][0, :2] = np.arange(1, 3)          # continues a sequence: one tap reaches back
        rng = np.random.default_rng(26)
        p["xinit"] = rng.standard_normal((1, 2, 3))
        gxf = rng.standard_normal((1, 2, 3))

        def loss():
            out, xf = O.conv1d_fwd(p["x"], p["w"], p["bias"], p["pos"], silu, lib=lib, xinit=p["xinit"],
                                   return_final=True)
            return float(np.sum(p["dout"] * out) + np.sum(gxf * xf))

        g = O.conv1d_bwd(p["x"], p["w"], p["bias"], p["pos"], p["dout"], silu, lib=lib,
                         xinit=p["xinit"], dxfinal=gxf)
        grads = {"x": g["dx"], "w": g["dw"], "bias": g["dbias"], "xinit": g["dxinit"]}
        _fd(loss, p, list(grads), grads, f"conv with states silu={silu}")


def pin_check_positions_continued(lib):
    pos = W.positions_from_lengths([[3, 5]], 8)
    pos[0, :3] = [4, 5, 6]
    assert O.check_positions(pos, lib=lib) == 0
    assert O.check_positions(pos, lib=lib, continued=True) == -1
    pos[0, 0] = -1
    assert O.check_positions(pos, lib=lib, continued=True) == 0


# cheapest first (the mutant test stops at the first pin that rejects a mutant)
ALL_PINS = [
    pin_check_positions, pin_len1_conv, pin_len1_scan, pin_cumsum, pin_closed_conv,
    pin_closed_scan, pin_states, pin_library_conv, pin_pui_conv, pin_pui_scan, pin_fd_conv,
    pin_fd_scan_plain, pin_fd_scan, pin_check_positions_continued, pin_split_conv, pin_split_scan,
    pin_fd_conv_states, pin_fd_scan_states,
]
