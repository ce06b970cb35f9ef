"""Plant plausible mistakes in a copy of the oracle (CPU only) and require a pin to catch each.

The mutated sources are written to a temporary directory; the real oracle is
untouched.  A mutant that no pin rejects would mean the pins leave that part of
the oracle unchecked.
"""
import os

import pytest

import oracle
import oracle_pins as P

SRC = open(oracle.SRC_PATH).read()

# (id, text in oracle.c, replacement, occurrence index or None for all)
MUTANTS = [
    ("conv-mask-off-by-one", "if (k > pr[l]) break;                       /* before", "if (k > pr[l] + 1) break;                       /* before", None),
    ("conv-mask-ignored", "if (k > pr[l]) break;                       /* before", "if (0) break;                       /* before", None),
    ("conv-taps-reversed", "acc += wd[width - 1 - k] * x_at(xr, xi, width, l - k);", "acc += wd[k] * x_at(xr, xi, width, l - k);", None),
    ("conv-bias-dropped", "double acc = b0;", "double acc = 0.0;", None),
    ("conv-silu-grad-sign", "g *= s * (1.0 + v * (1.0 - s));", "g *= s * (1.0 - v * (1.0 - s));", None),
    ("conv-dx-tap", "dxr[l - k] += wd[width - 1 - k] * g;", "dxr[l - k] += wd[k] * g;", None),
    ("conv-dw-index", "dwd[width - 1 - k] += g * x_at(xr, xi, width, l - k);", "dwd[width - 1 - k] += g * x_at(xr, xi, width, l);", None),
    ("conv-bwd-mask", "if (k > pr[l]) break;\n                    if (l - k >= 0)", "if (0) break;\n                    if (l - k >= 0)", None),
    ("conv-xinit-ignored", "return xi ? xi[width - 1 + m] : 0.0;", "return 0.0;", None),
    ("conv-xinit-reversed", "return xi ? xi[width - 1 + m] : 0.0;", "return xi ? xi[-1 - m] : 0.0;", None),
    ("conv-xfinal-offset", "x_at(xr, xi, width, seqlen - (width - 1) + i)", "x_at(xr, xi, width, seqlen - width + i)", None),
    ("conv-dxinit-missing", "dxi[width - 1 + l - k] += wd[width - 1 - k] * g;", ";", None),
    ("conv-dxfinal-ignored", "if (m >= 0) dxr[m] += gf;", "if (m >= 0) dxr[m] += 0.0;", None),
    ("scan-reset-missing", "const double a = (pr[l] == 0) ? 0.0 : exp(dt * A[d * N + n]);", "const double a = exp(dt * A[d * N + n]);", None),
    ("scan-reset-wrong-index", "const double a = (pr[l] == 0) ? 0.0 : exp(dt * A[d * N + n]);", "const double a = (pr[l] == 1) ? 0.0 : exp(dt * A[d * N + n]);", None),
    ("scan-rowfwd-reset-missing", "const double a = (pr[l] == 0) ? 0.0 : exp(dt * Ad[n]);", "const double a = exp(dt * Ad[n]);", None),
    ("scan-decay-sign", "const double a = (pr[l] == 0) ? 0.0 : exp(dt * A[d * N + n]);", "const double a = (pr[l] == 0) ? 0.0 : exp(-dt * A[d * N + n]);", None),
    ("scan-rowfwd-decay-sign", "exp(dt * Ad[n]);", "exp(-dt * Ad[n]);", None),
    ("scan-bx-drops-dt", "h[n] = a * h[n] + dt * Bb[(int64_t)n * seqlen + l] * ur[l];\n                        y +=", "h[n] = a * h[n] + Bb[(int64_t)n * seqlen + l] * ur[l];\n                        y +=", None),
    ("scan-rowfwd-bx-drops-dt", "h[n] = a * h[n] + dt * Bb[(int64_t)n * seqlen + l] * ur[l];\n            if (as_)", "h[n] = a * h[n] + Bb[(int64_t)n * seqlen + l] * ur[l];\n            if (as_)", None),
    ("scan-D-dropped", "const double yD = y + (D ? D[d] * ur[l] : 0.0);\n                    out[", "const double yD = y;\n                    out[", None),
    ("scan-gate-sigmoid-only", "out[row + l] = z ? yD * z[row + l] * sigmoid(z[row + l]) : yD;", "out[row + l] = z ? yD * sigmoid(z[row + l]) : yD;", None),
    ("scan-softplus-missing", "return sp ? softplus(s) : s;", "return s;", None),
    ("scan-fwd-h0-ignored", "h[n] = h0 ? h0[(b * dim + d) * N + n] : 0.0;", "h[n] = 0.0;", None),
    ("scan-rowfwd-h0-ignored", "h[n] = h0 ? h0[n] : 0.0;", "h[n] = 0.0;", None),
    ("scan-bwd-reverse-no-decay", "dh[n] = dy[l] * Cb[(int64_t)n * seqlen + l] + an * dh[n];", "dh[n] = dy[l] * Cb[(int64_t)n * seqlen + l] + dh[n];", None),
    ("scan-bwd-reverse-wrong-multiplier", "const double an = (l + 1 < seqlen) ? as_[(l + 1) * N + n] : 1.0;", "const double an = as_[l * N + n];", None),
    ("scan-bwd-reverse-reset-ignored", "const double an = (l + 1 < seqlen) ? as_[(l + 1) * N + n] : 1.0;", "const double an = (l + 1 < seqlen) ? exp(dts[l + 1] * A[d * N + n]) : 1.0;", None),
    ("scan-bwd-dhfinal-ignored", "dh[n] = dhfinal ? dhfinal[(b * dim + d) * N + n] : 0.0;", "dh[n] = 0.0;", None),
    ("scan-bwd-dA-sign", "ddt[l] += t * A[d * N + n];", "ddt[l] -= t * A[d * N + n];", None),
    ("scan-bwd-dA-prev-state", "const double hp = l > 0 ? hs[(l - 1) * N + n] : (h0r ? h0r[n] : 0.0);", "const double hp = hs[l * N + n];", None),
    ("scan-bwd-h0-term-missing", "(h0r ? h0r[n] : 0.0);", "0.0;", None),
    ("scan-bwd-dh0-no-multiplier", "= as_[n] * dh[n];", "= dh[n];", None),
    ("scan-bwd-dB-transposed", "dBb[(int64_t)n * seqlen + l] += dh[n] * dt * ur[l];", "dBb[(int64_t)n * seqlen + l] += dh[n] * ur[l];", None),
    ("scan-bwd-dC", "dCb[(int64_t)n * seqlen + l] += dyD * hs[l * N + n];", "dCb[(int64_t)n * seqlen + l] += g * hs[l * N + n];", None),
    ("scan-bwd-dz", "dz[row + l] = g * yD * s * (1.0 + zz * (1.0 - s));", "dz[row + l] = g * yD * s;", None),
    ("scan-bwd-softplus-grad", "gs = softplus_grad(dr[l] + (delta_bias ? delta_bias[d] : 0.0));", "gs = 1.0;", None),
    ("scan-bwd-du-missing-dt", "du[row + l] += dh[n] * dt * Bl;", "du[row + l] += dh[n] * Bl;", None),
    ("scan-bwd-dD", "if (D) dDd += dyD * ur[l];", "if (D) dDd += g * ur[l];", None),
    ("check-positions-start", "(continued ? pr[l] >= 0 : pr[l] == 0)", "(1)", None),
    ("check-positions-continued-negative", "(continued ? pr[l] >= 0 : pr[l] == 0)", "(continued ? 1 : pr[l] == 0)", None),
]


@pytest.mark.parametrize("mid,old,new,occ", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_reject_mutant(mid, old, new, occ, tmp_path):
    assert old in SRC, f"mutation target for {mid} not found in oracle.c"
    src = SRC.replace(old, new)
    path = tmp_path / "oracle_mut.c"
    path.write_text(src)
    lib_path = str(tmp_path / f"liboracle_{mid}.so")
    oracle.build(src=str(path), out=lib_path)
    lib = oracle.load(lib_path)
    oracle.set_num_threads(1, lib=lib)       # tiny problems; avoid oversubscribing xdist workers
    caught = None
    for pin in P.ALL_PINS:                   # cheapest pins first; stop at the first rejection
        try:
            pin(lib)
        except (AssertionError, FloatingPointError, ValueError) as e:
            caught = (pin.__name__, str(e)[:120])
            break
    assert caught, f"no pin caught mutant {mid}"
