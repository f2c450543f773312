"""Planted mistakes in copies of the CPU oracle must each fail a pin.

Every mutant below is a plausible slip in transcribing the paper (a flipped
sign or swapped index in eq. 3 or eq. 7, the operands of the Hamilton product
swapped, a wrong padding or dilation term, an unbiased variance, eps outside
the square root, an untransposed Jacobian in a gradient, a dropped factor of
the Poincare map, ...).  Each is compiled from a text substitution of quan_oracle.c into a
temporary library and run through the pins of oracle_pins.py; the test passes
only if at least one pin rejects it.  All mutations stay in bounds."""
import os

import pytest

import oracle
from oracle import build as obuild
from oracle_pins import ALL_PINS

SRC = open(obuild.SRC).read()

MUTANTS = [
    # eq. 3: one sign flipped in each output component
    ("sign r", "out[0] = pr * qr - pi * qi", "out[0] = pr * qr + pi * qi"),
    ("sign r2", "- pj * qj - pk * qk", "- pj * qj + pk * qk"),
    ("sign i", "out[1] = pr * qi + pi * qr", "out[1] = pr * qi - pi * qr"),
    ("sign i2", "+ pj * qk - pk * qj", "- pj * qk - pk * qj"),
    ("sign j", "out[2] = pr * qj - pi * qk", "out[2] = pr * qj + pi * qk"),
    ("sign j2", "+ pj * qr + pk * qi", "+ pj * qr - pk * qi"),
    ("sign k", "out[3] = pr * qk + pi * qj", "out[3] = pr * qk - pi * qj"),
    ("sign k2", "- pj * qi + pk * qr", "+ pj * qi + pk * qr"),
    # eq. 3: a dropped term, a wrong component index
    ("dropped term", "- pj * qj - pk * qk;", "- pj * qj;"),
    ("wrong index", "out[1] = pr * qi + pi * qr + pj * qk", "out[1] = pr * qi + pi * qr + pj * qj"),
    # right instead of left multiplication (X (x) W)
    ("operands swapped", "quan_oracle_hamilton(wv, xv, prod);", "quan_oracle_hamilton(xv, wv, prod);"),
    # convolution indexing
    ("pad sign", "\n                            const int64_t iy = oy * sh - ph + ky * dh;", "\n                            const int64_t iy = oy * sh + ph + ky * dh;"),
    ("no dilation", "\n                                const int64_t ix = ox * sw - pw + kx * dw;", "\n                                const int64_t ix = ox * sw - pw + kx;"),
    ("stride dropped", "\n                            const int64_t iy = oy * sh - ph + ky * dh;", "\n                            const int64_t iy = oy - ph + ky * dh;"),
    ("kernel flipped", "const int64_t widx = ((o * Cin + c) * KH + ky) * KW + kx;",
     "const int64_t widx = ((o * Cin + c) * KH + (KH - 1 - ky)) * KW + (KW - 1 - kx);"),
    ("ky/kx swapped", "const int64_t widx = ((o * Cin + c) * KH + ky) * KW + kx;",
     "const int64_t widx = ((o * Cin + c) * KH + kx) * KW + ky;"),
    ("output permuted", "y[((n * 4 * Cout + q * Cout + o) * Ho + oy) * Wo + ox]",
     "y[((n * 4 * Cout + o * 4 + q) * Ho + oy) * Wo + ox]"),
    ("bias one comp", "acc[q] = bias[q * Cout + o];", "acc[q] = bias[o];"),
    # IQBN
    ("unbiased var", "const double sigma2 = ss / cnt;", "const double sigma2 = ss / (cnt - 1.0);"),
    ("eps outside sqrt", "1.0 / sqrt(sigma2 + eps)", "1.0 / (sqrt(sigma2) + eps)"),
    ("gamma/beta swapped", "double v = (xs[t] - mu) * inv * g + b;\n                    if (relu && v < 0.0)\n                        v = 0.0;\n                    os[t] = v;\n                }\n            }\n            if (mean)",
     "double v = (xs[t] - mu) * inv * b + g;\n                    if (relu && v < 0.0)\n                        v = 0.0;\n                    os[t] = v;\n                }\n            }\n            if (mean)"),
    ("std not var", "1.0 / sqrt(sigma2 + eps)", "1.0 / (sigma2 + eps)"),
    ("relu inverted", "if (relu && v < 0.0)\n                        v = 0.0;\n                    os[t] = v;\n                }\n            }\n            if (mean)",
     "if (relu && v > 0.0)\n                        v = 0.0;\n                    os[t] = v;\n                }\n            }\n            if (mean)"),
    # separable convolution (eq. 7)
    ("eq. 7 sign", "{1.0, 1.0, 1.0, -1.0},   /* y_i", "{1.0, 1.0, -1.0, -1.0},   /* y_i"),
    ("eq. 7 rows swapped", "{1.0, -1.0, 1.0, 1.0},   /* y_j", "{1.0, 1.0, -1.0, 1.0},   /* y_j"),
    ("eq. 7 cross term", "conv[q] += w[q * wq + ((o * Cin + c) * KH + ky) * KW + kx] *\n                                               x[q * xq",
     "conv[q] += w[((q + 1) & 3) * wq + ((o * Cin + c) * KH + ky) * KW + kx] *\n                                               x[q * xq"),
    ("eq. 7 bias dropped", "double v = bias ? bias[p * Cout + o] : 0.0;", "double v = bias ? 0.0 * bias[p * Cout + o] : 0.0;"),
    # conv gradients
    ("dX Jacobian not transposed", "s += L[p][q] * g[p];", "s += L[q][p] * g[p];"),
    ("dW Jacobian not transposed", "s += R[p][q] * g[p];", "s += R[q][p] * g[p];"),
    ("dW uses the left matrix", "quan_oracle_hamilton(e, q, col);", "quan_oracle_hamilton(q, e, col);"),
    ("dX stride dropped", "const int64_t iy = oy * sh - ph + ky * dh;\n                                if (iy < 0 || iy >= H)\n                                    continue;\n                                for (int64_t kx = 0; kx < KW; ++kx) {\n                                    const int64_t ix = ox * sw - pw + kx * dw;\n                                    if (ix < 0 || ix >= W)\n                                        continue;\n                                    double wv[4], L[4][4];",
     "const int64_t iy = oy - ph + ky * dh;\n                                if (iy < 0 || iy >= H)\n                                    continue;\n                                for (int64_t kx = 0; kx < KW; ++kx) {\n                                    const int64_t ix = ox * sw - pw + kx * dw;\n                                    if (ix < 0 || ix >= W)\n                                        continue;\n                                    double wv[4], L[4][4];"),
    ("dbias one component", "s += dy[n * 4 * yq + q * yq + o * Ho * Wo + t];", "s += dy[n * 4 * yq + o * Ho * Wo + t];"),
    # separable conv gradients (eqs. 8-10)
    ("M transposed", "z[q] += kMixing[q][p] * dy[n * 4 * yq + p * yq + (o * Ho + oy) * Wo + ox];\n                        }\n                        for (int q = 0; q < 4; ++q)\n                            for (int64_t c = 0; c < Cin; ++c)\n                                for (int64_t ky = 0; ky < KH; ++ky) {\n                                    const int64_t iy = oy * sh - ph + ky * dh;\n                                    if (iy < 0 || iy >= H)\n                                        continue;\n                                    for (int64_t kx = 0; kx < KW; ++kx) {\n                                        const int64_t ix = ox * sw - pw + kx * dw;\n                                        if (ix < 0 || ix >= W)\n                                            continue;\n                                        dx[",
     "z[q] += kMixing[p][q] * dy[n * 4 * yq + p * yq + (o * Ho + oy) * Wo + ox];\n                        }\n                        for (int q = 0; q < 4; ++q)\n                            for (int64_t c = 0; c < Cin; ++c)\n                                for (int64_t ky = 0; ky < KH; ++ky) {\n                                    const int64_t iy = oy * sh - ph + ky * dh;\n                                    if (iy < 0 || iy >= H)\n                                        continue;\n                                    for (int64_t kx = 0; kx < KW; ++kx) {\n                                        const int64_t ix = ox * sw - pw + kx * dw;\n                                        if (ix < 0 || ix >= W)\n                                            continue;\n                                        dx["),
    ("M sign", "{-1.0, 1.0, 1.0, -1.0},\n    {-1.0, -1.0, 1.0, 1.0},\n};", "{-1.0, 1.0, -1.0, -1.0},\n    {-1.0, -1.0, 1.0, 1.0},\n};"),
    ("separable dX wrong kernel", "w[q * wq + ((o * Cin + c) * KH + ky) * KW + kx] * z[q];", "w[((q + 1) & 3) * wq + ((o * Cin + c) * KH + ky) * KW + kx] * z[q];"),
    ("separable dW unmixed", "x[n * 4 * xq + q * xq + (c * H + iy) * W + ix] * z[q];", "x[n * 4 * xq + q * xq + (c * H + iy) * W + ix] * dy[n * 4 * yq + q * yq + (o * Ho + oy) * Wo + ox];"),
    ("separable dX kernel not flipped back", "dx[n * 4 * xq + q * xq + (c * H + iy) * W + ix] +=\n                                            w[q * wq + ((o * Cin + c) * KH + ky) * KW + kx] * z[q];",
     "dx[n * 4 * xq + q * xq + (c * H + iy) * W + ix] +=\n                                            w[q * wq + ((o * Cin + c) * KH + (KH - 1 - ky)) * KW + (KW - 1 - kx)] * z[q];"),
    # IQBN inference and backward
    ("inference eps outside sqrt", "const double inv = 1.0 / sqrt(var[q * C + c] + eps);",
     "const double inv = 1.0 / (sqrt(var[q * C + c]) + eps);"),
    ("inference mean ignored", "double v = (xs[t] - mu) * inv * g + b;\n                    if (relu && v < 0.0)\n                        v = 0.0;\n                    os[t] = v;\n                }\n            }\n        }\n    }",
     "double v = (xs[t] - 0.0 * mu) * inv * g + b;\n                    if (relu && v < 0.0)\n                        v = 0.0;\n                    os[t] = v;\n                }\n            }\n        }\n    }"),
    ("backward xhat term dropped", "dx[idx] = ga / sd * (g - sg / cnt - xhat * sgx / cnt);", "dx[idx] = ga / sd * (g - sg / cnt);"),
    ("backward mean term dropped", "dx[idx] = ga / sd * (g - sg / cnt - xhat * sgx / cnt);", "dx[idx] = ga / sd * (g - xhat * sgx / cnt);"),
    ("backward relu mask ignored", "if (relu && !(ga * xhat + be > 0.0))\n                        g = 0.0;\n                    dx[idx]",
     "if (0 && relu && !(ga * xhat + be > 0.0))\n                        g = 0.0;\n                    dx[idx]"),
    ("backward unbiased var", "const double sd = sqrt(s2 / cnt + eps);", "const double sd = sqrt(s2 / (cnt - 1.0) + eps);"),
    # Poincare mapping (eq. 4)
    ("poincare factor 2 dropped", "q[(n * 4 + 1) * hw + t] = 2.0 * r / den;", "q[(n * 4 + 1) * hw + t] = r / den;"),
    ("poincare g/b swapped", "q[(n * 4 + 2) * hw + t] = 2.0 * g / den;", "q[(n * 4 + 2) * hw + t] = 2.0 * b / den;"),
    ("poincare real part sign", "q[(n * 4 + 0) * hw + t] = (1.0 - n2) / den;", "q[(n * 4 + 0) * hw + t] = (n2 - 1.0) / den;"),
    ("shared stats across components", "const double *xs = x + (n * 4 * C + q * C + c) * hw;\n                for (int64_t t = 0; t < hw; ++t)\n                    s += xs[t];",
     "const double *xs = x + (n * 4 * C + 0 * C + c) * hw;\n                for (int64_t t = 0; t < hw; ++t)\n                    s += xs[t];"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new):
    assert SRC.count(old) == 1, f"mutation anchor not unique/found: {old!r}"
    src = tmp_path / "mutant.c"
    src.write_text(SRC.replace(old, new))
    lib = obuild.build(str(src), str(tmp_path / "libmutant.so"))
    orc = oracle.Oracle(lib)
    failed = []
    for pin in ALL_PINS:
        try:
            pin(orc)
        except AssertionError:
            failed.append(pin.__name__)
            break
    assert failed, f"mutant '{name}' passed every pin"


def test_unmutated_copy_passes(tmp_path):
    src = tmp_path / "copy.c"
    src.write_text(SRC)
    orc = oracle.Oracle(obuild.build(str(src), str(tmp_path / "libcopy.so")))
    for pin in ALL_PINS:
        pin(orc)
