"""Checks that pin the CPU oracle to what the paper and the mathematics fix.

Each ``pin_*`` function takes an ``oracle.Oracle`` and raises AssertionError if
the oracle disagrees with an independent source of truth:

  * the paper's printed relations and tables (``tests/golden``): the unit
    relations of eq. 2, the expansion of eq. 5, the Hamilton matrix of eq. 6,
    the separable form of eq. 7 and the mixing matrix printed with eq. 9;
  * an independent construction of the quaternion algebra (2x2 complex
    matrices, themselves checked against eq. 2);
  * closed forms and invariants (identity kernel, multiplicative norm,
    conjugate = transpose, associativity, linearity, IQBN moments, adjoint
    identities of the gradients, unit norm and inverse of the Poincare map);
  * special cases that reduce to library routines (torch's fp64 conv2d,
    batch_norm and autograd, numpy's complex arithmetic, numpy mean/var).

The same checks run against deliberately broken builds of the oracle in
test_oracle_mutants.py, to show that each plausible mistake fails one of them.
"""
import functools
import os

import numpy as np
import torch
import torch.nn.functional as F

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
COMP = {"r": 0, "i": 1, "j": 2, "k": 3}
UNIT = {"1": np.array([1.0, 0, 0, 0]), "i": np.array([0, 1.0, 0, 0]),
        "j": np.array([0, 0, 1.0, 0]), "k": np.array([0, 0, 0, 1.0])}


def _lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [ln.strip() for ln in f if ln.strip() and not ln.startswith("#")]


def eq2_relations():
    """[(['i','j','k'], -1.0), ...] from the eq. 2 fixture."""
    rel = []
    for ln in _lines("unit_relations_eq2.txt"):
        lhs, rhs = [s.strip() for s in ln.split("=")]
        rel.append((lhs.split("*"), float(rhs)))
    return rel


def eq5_coefficients():
    """C[p, a, b]: coefficient of W_a * X_b in output component p (eq. 5)."""
    C = np.zeros((4, 4, 4))
    for ln in _lines("hamilton_expansion_eq5.txt"):
        head, terms = ln.split(":")
        p = COMP[head.strip()]
        for t in terms.split():
            sign = -1.0 if t[0] == "-" else 1.0
            wpart, xpart = t[1:].split("*")
            C[p, COMP[wpart.split("_")[1]], COMP[xpart.split("_")[1]]] += sign
    return C


def eq6_matrix_pattern():
    """(sign[p, q], comp[p, q]): entry (p, q) of eq. 6 is sign * w_comp."""
    sign = np.zeros((4, 4))
    comp = np.zeros((4, 4), dtype=int)
    for p, ln in enumerate(_lines("hamilton_matrix_eq6.txt")):
        for q, tok in enumerate(ln.split()):
            sign[p, q] = -1.0 if tok.startswith("-") else 1.0
            comp[p, q] = COMP[tok.lstrip("-").split("_")[1]]
    return sign, comp


def eq6_matrix(w):
    sign, comp = eq6_matrix_pattern()
    return sign * np.asarray(w, dtype=np.float64)[comp]


# --- independent model of the quaternion algebra: 2x2 complex matrices ------

def crep(q):
    """r + i i + j j + k k  ->  [[r + i*1j, j + k*1j], [-j + k*1j, r - i*1j]]."""
    r, i, j, k = np.moveaxis(np.asarray(q, dtype=np.float64), -1, 0)
    top = np.stack([r + 1j * i, j + 1j * k], axis=-1)
    bot = np.stack([-j + 1j * k, r - 1j * i], axis=-1)
    return np.stack([top, bot], axis=-2)


def cunrep(m):
    return np.stack([m[..., 0, 0].real, m[..., 0, 0].imag,
                     m[..., 0, 1].real, m[..., 0, 1].imag], axis=-1)


def cprod(p, q):
    """Quaternion product through the complex-matrix model."""
    return cunrep(crep(p) @ crep(q))


def brute_qconv_crep(x, w, bias, stride, pad, dil):
    """Quaternion convolution summed tap by tap through the complex-matrix
    model (numpy complex arithmetic only).  x [N,4,Cin,H,W], w [4,Cout,Cin,k,k]."""
    N, _, Cin, H, W = x.shape
    Cout, KH, KW = w.shape[1], w.shape[3], w.shape[4]
    Ho = (H + 2 * pad - dil * (KH - 1) - 1) // stride + 1
    Wo = (W + 2 * pad - dil * (KW - 1) - 1) // stride + 1
    xr = crep(np.moveaxis(x, 1, -1))          # [N,Cin,H,W,2,2]
    wr = crep(np.moveaxis(w, 0, -1))          # [Cout,Cin,KH,KW,2,2]
    y = np.zeros((N, Cout, Ho, Wo, 2, 2), dtype=np.complex128)
    for oy in range(Ho):
        for ox in range(Wo):
            for ky in range(KH):
                iy = oy * stride - pad + ky * dil
                if iy < 0 or iy >= H:
                    continue
                for kx in range(KW):
                    ix = ox * stride - pad + kx * dil
                    if ix < 0 or ix >= W:
                        continue
                    # sum over c of W[o,c] * X[n,c]  -> [N, Cout, 2, 2]
                    prod = wr[None, :, :, ky, kx] @ xr[:, None, :, iy, ix]
                    y[:, :, oy, ox] += prod.sum(axis=2)
    out = np.moveaxis(cunrep(y), -1, 1)       # [N,4,Cout,Ho,Wo]
    if bias is not None:
        out = out + np.asarray(bias)[None, :, :, None, None]
    return out


def block_weight(w):
    """Real [4*Cout, 4*Cin, k, k] weight from the eq. 6 sign/component pattern:
    block (p, q) = sign[p, q] * W_comp[p, q]."""
    sign, comp = eq6_matrix_pattern()
    w = np.asarray(w, dtype=np.float64)
    rows = [np.concatenate([sign[p, q] * w[comp[p, q]] for q in range(4)], axis=1)
            for p in range(4)]
    return np.concatenate(rows, axis=0)


def torch_block_conv(x, w, bias, stride, pad, dil):
    N, _, Cin, H, W = x.shape
    Cout = w.shape[1]
    xt = torch.from_numpy(np.ascontiguousarray(x.reshape(N, 4 * Cin, H, W)))
    wt = torch.from_numpy(block_weight(w))
    bt = None if bias is None else torch.from_numpy(np.asarray(bias, np.float64).reshape(-1))
    y = F.conv2d(xt, wt, bt, stride=stride, padding=pad, dilation=dil).numpy()
    return y.reshape(N, 4, Cout, y.shape[2], y.shape[3])


def _rng(seed):
    return np.random.default_rng(seed)


def _close(a, b, tol=1e-12, what=""):
    a, b = np.asarray(a), np.asarray(b)
    scale = max(1.0, float(np.max(np.abs(b))) if b.size else 1.0)
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert err <= tol * scale, f"{what}: max abs err {err:.3e} (scale {scale:.3e})"


# ----------------------------- Hamilton product ------------------------------

def pin_eq2_unit_relations(orc):
    """Every relation of eq. 2 holds for the oracle's product."""
    for units, value in eq2_relations():
        prod = functools.reduce(orc.hamilton, [UNIT[u] for u in units])
        _close(prod, value * UNIT["1"], 0, f"eq. 2: {'*'.join(units)}")


def pin_unit_table_derived(orc):
    """Consequences of eq. 2: ij = k, jk = i, ki = j and anticommutation."""
    for a, b, c in [("i", "j", "k"), ("j", "k", "i"), ("k", "i", "j")]:
        _close(orc.hamilton(UNIT[a], UNIT[b]), UNIT[c], 0, f"{a}{b}")
        _close(orc.hamilton(UNIT[b], UNIT[a]), -UNIT[c], 0, f"{b}{a}")
    for u in "1ijk":
        _close(orc.hamilton(UNIT["1"], UNIT[u]), UNIT[u], 0, f"1{u}")
        _close(orc.hamilton(UNIT[u], UNIT["1"]), UNIT[u], 0, f"{u}1")


def pin_complex_model(orc):
    """The product agrees with the 2x2 complex-matrix model of the algebra
    (which itself satisfies eq. 2) on random quaternions."""
    for units, value in eq2_relations():
        m = functools.reduce(lambda a, b: a @ b, [crep(UNIT[u]) for u in units])
        assert np.allclose(m, value * np.eye(2)), "complex model breaks eq. 2"
    rng = _rng(11)
    for _ in range(50):
        p, q = rng.standard_normal(4), rng.standard_normal(4)
        _close(orc.hamilton(p, q), cprod(p, q), 1e-14, "complex model")


def pin_eq6_matrix(orc):
    """p (x) q equals the eq. 6 matrix of p times the column q."""
    rng = _rng(12)
    for _ in range(50):
        p, q = rng.standard_normal(4), rng.standard_normal(4)
        _close(orc.hamilton(p, q), eq6_matrix(p) @ q, 1e-14, "eq. 6")


# --------------------------- quaternion convolution ---------------------------

def _conv_unit(orc, wq, xq):
    """1x1 conv, one channel, one pixel: W = wq, X = xq."""
    x = np.asarray(xq, dtype=np.float64).reshape(1, 4, 1, 1, 1)
    w = np.asarray(wq, dtype=np.float64).reshape(4, 1, 1, 1, 1)
    return orc.qconv2d(x, w).reshape(4)


def pin_eq5_expansion(orc):
    """Each basis pair (W = e_a, X = e_b) produces the eq. 5 coefficients."""
    C = eq5_coefficients()
    for a in range(4):
        for b in range(4):
            ea, eb = np.eye(4)[a], np.eye(4)[b]
            _close(_conv_unit(orc, ea, eb), C[:, a, b], 0, f"eq. 5 W_{a} X_{b}")


def pin_orientation(orc):
    """The kernel multiplies from the left: W = i, X = j gives +k (X (x) W = -k)."""
    _close(_conv_unit(orc, UNIT["i"], UNIT["j"]), UNIT["k"], 0, "W=i, X=j")
    _close(_conv_unit(orc, UNIT["j"], UNIT["i"]), -UNIT["k"], 0, "W=j, X=i")


def pin_identity_kernel(orc):
    """W_r = delta (centre tap, o == c), W_i = W_j = W_k = 0 returns the input."""
    rng = _rng(13)
    for k in (1, 3, 5):
        x = rng.standard_normal((2, 4, 3, 7, 5))
        w = np.zeros((4, 3, 3, k, k))
        for c in range(3):
            w[0, c, c, k // 2, k // 2] = 1.0
        _close(orc.qconv2d(x, w, None, 1, k // 2, 1), x, 0, f"identity k={k}")


def pin_norm(orc):
    """|W (x) X| = |W| |X| per pixel for a 1x1, single-channel convolution."""
    rng = _rng(14)
    w = rng.standard_normal((4, 1, 1, 1, 1))
    x = rng.standard_normal((3, 4, 1, 5, 6))
    y = orc.qconv2d(x, w)
    ny = np.linalg.norm(y, axis=1)
    nx = np.linalg.norm(x, axis=1)
    _close(ny, np.linalg.norm(w) * nx, 1e-13, "norm")


def pin_conjugate_adjoint(orc):
    """<W (x) X, Y> = <X, conj(W) (x) Y>: the Hamilton matrix of the conjugate
    is the transpose, for a 1x1, single-channel convolution."""
    rng = _rng(15)
    w = rng.standard_normal(4)
    wbar = w * np.array([1, -1, -1, -1])
    x = rng.standard_normal((2, 4, 1, 3, 3))
    yv = rng.standard_normal((2, 4, 1, 3, 3))
    lhs = np.sum(orc.qconv2d(x, w.reshape(4, 1, 1, 1, 1)) * yv)
    rhs = np.sum(x * orc.qconv2d(yv, wbar.reshape(4, 1, 1, 1, 1)))
    _close(lhs, rhs, 1e-12, "adjoint")


def pin_real_reduction(orc):
    """W_i = W_j = W_k = 0: every component is the real convolution with W_r
    (torch fp64 conv2d), over a stride/pad/dilation sweep."""
    rng = _rng(16)
    for (k, s, p, d) in [(3, 1, 1, 1), (3, 2, 1, 1), (5, 1, 2, 2), (1, 1, 0, 1), (3, 2, 0, 2)]:
        x = rng.standard_normal((2, 4, 3, 9, 8))
        w = np.zeros((4, 5, 3, k, k))
        w[0] = rng.standard_normal((5, 3, k, k))
        y = orc.qconv2d(x, w, None, s, p, d)
        for q in range(4):
            ref = F.conv2d(torch.from_numpy(np.ascontiguousarray(x[:, q])),
                           torch.from_numpy(w[0]), stride=s, padding=p, dilation=d).numpy()
            _close(y[:, q], ref, 1e-13, f"real reduction q={q} k={k} s={s} p={p} d={d}")


def pin_complex_reduction(orc):
    """X_j = X_k = 0 and W_j = W_k = 0: (Y_r, Y_i) is the complex convolution
    (numpy complex128) and Y_j = Y_k = 0."""
    rng = _rng(17)
    N, Cin, Cout, H, W, k, s, p = 2, 3, 2, 6, 7, 3, 1, 1
    x = np.zeros((N, 4, Cin, H, W))
    x[:, :2] = rng.standard_normal((N, 2, Cin, H, W))
    w = np.zeros((4, Cout, Cin, k, k))
    w[:2] = rng.standard_normal((2, Cout, Cin, k, k))
    y = orc.qconv2d(x, w, None, s, p, 1)
    xc = x[:, 0] + 1j * x[:, 1]
    wc = w[0] + 1j * w[1]
    xp = np.pad(xc, ((0, 0), (0, 0), (p, p), (p, p)))
    ref = np.zeros((N, Cout, H, W), dtype=np.complex128)
    for ky in range(k):
        for kx in range(k):
            patch = xp[:, :, ky:ky + H, kx:kx + W]           # [N,Cin,H,W]
            ref += np.einsum("oc,nchw->nohw", wc[:, :, ky, kx], patch)
    _close(y[:, 0], ref.real, 1e-13, "complex reduction real")
    _close(y[:, 1], ref.imag, 1e-13, "complex reduction imag")
    _close(y[:, 2:], np.zeros_like(y[:, 2:]), 0, "complex reduction j,k")


CONV_SWEEP = [
    # (N, Cin, Cout, H, W, k, stride, pad, dil)
    (2, 3, 5, 7, 9, 3, 1, 1, 1),
    (1, 2, 3, 9, 7, 3, 2, 1, 1),
    (2, 3, 2, 8, 11, 5, 1, 2, 1),
    (1, 4, 4, 10, 9, 3, 2, 2, 2),
    (2, 2, 3, 6, 5, 1, 1, 0, 1),
    (1, 3, 2, 7, 8, 3, 1, 0, 2),
    (1, 1, 2, 5, 5, 5, 2, 1, 1),
]


def pin_block_matrix(orc):
    """Agreement with torch's fp64 conv2d of the real 4Cin -> 4Cout block
    weight built from the eq. 6 pattern, with bias, over a shape sweep."""
    rng = _rng(18)
    for (N, Cin, Cout, H, W, k, s, p, d) in CONV_SWEEP:
        x = rng.standard_normal((N, 4, Cin, H, W))
        w = rng.standard_normal((4, Cout, Cin, k, k))
        b = rng.standard_normal((4, Cout))
        y = orc.qconv2d(x, w, b, s, p, d)
        ref = torch_block_conv(x, w, b, s, p, d)
        _close(y, ref, 1e-12, f"block matrix {(N, Cin, Cout, H, W, k, s, p, d)}")


def pin_brute_force_complex_model(orc):
    """Tap-by-tap quaternion convolution through the complex-matrix model."""
    rng = _rng(19)
    for (N, Cin, Cout, H, W, k, s, p, d) in CONV_SWEEP[:4]:
        x = rng.standard_normal((N, 4, Cin, H, W))
        w = rng.standard_normal((4, Cout, Cin, k, k))
        b = rng.standard_normal((4, Cout))
        y = orc.qconv2d(x, w, b, s, p, d)
        _close(y, brute_qconv_crep(x, w, b, s, p, d), 1e-12, "complex-model brute force")


def pin_associativity(orc):
    """Two chained 1x1 layers A then B equal one layer whose weight is the
    quaternion matrix product sum_m B[o,m] (x) A[m,c] (complex model)."""
    rng = _rng(20)
    Cin, Cm, Cout = 3, 4, 2
    A = rng.standard_normal((4, Cm, Cin, 1, 1))
    B = rng.standard_normal((4, Cout, Cm, 1, 1))
    x = rng.standard_normal((2, 4, Cin, 4, 5))
    y2 = orc.qconv2d(orc.qconv2d(x, A), B)
    Aq = np.moveaxis(A[..., 0, 0], 0, -1)        # [Cm, Cin, 4]
    Bq = np.moveaxis(B[..., 0, 0], 0, -1)        # [Cout, Cm, 4]
    Cq = np.zeros((Cout, Cin, 4))
    for o in range(Cout):
        for c in range(Cin):
            for m in range(Cm):
                Cq[o, c] += cprod(Bq[o, m], Aq[m, c])
    Cw = np.moveaxis(Cq, -1, 0)[..., None, None]
    _close(y2, orc.qconv2d(x, Cw), 1e-12, "associativity")


def pin_linearity(orc):
    """conv is linear in X and in W."""
    rng = _rng(21)
    x1, x2 = rng.standard_normal((2, 2, 4, 3, 6, 5))
    w1, w2 = rng.standard_normal((2, 4, 2, 3, 3, 3))
    a, b = 0.7, -1.3
    _close(orc.qconv2d(a * x1 + b * x2, w1, None, 1, 1),
           a * orc.qconv2d(x1, w1, None, 1, 1) + b * orc.qconv2d(x2, w1, None, 1, 1), 1e-12, "lin X")
    _close(orc.qconv2d(x1, a * w1 + b * w2, None, 1, 1),
           a * orc.qconv2d(x1, w1, None, 1, 1) + b * orc.qconv2d(x1, w2, None, 1, 1), 1e-12, "lin W")


def pin_bias(orc):
    """The bias is one quaternion per output channel, added after the sum."""
    rng = _rng(22)
    x = rng.standard_normal((2, 4, 2, 5, 5))
    w = rng.standard_normal((4, 3, 2, 3, 3))
    b = rng.standard_normal((4, 3))
    _close(orc.qconv2d(x, w, b, 1, 1), orc.qconv2d(x, w, None, 1, 1) + b[None, :, :, None, None],
           1e-13, "bias")


# ------------------------------------ IQBN ------------------------------------

def pin_iqbn_batch_norm(orc):
    """IQBN equals torch's fp64 training-mode batch_norm over the 4C real
    channels (each component/channel pair normalised on its own)."""
    rng = _rng(23)
    for (N, C, H, W) in [(4, 3, 5, 6), (2, 1, 1, 7), (3, 2, 4, 4)]:
        x = rng.standard_normal((N, 4, C, H, W)) * 3.0 + rng.standard_normal((1, 4, C, 1, 1))
        g = rng.uniform(0.5, 1.5, (4, C))
        b = rng.standard_normal((4, C))
        for relu in (False, True):
            out, mean, var = orc.iqbn(x, g, b, 1e-5, relu)
            ref = F.batch_norm(torch.from_numpy(x.reshape(N, 4 * C, H, W)), None, None,
                               torch.from_numpy(g.reshape(-1)), torch.from_numpy(b.reshape(-1)),
                               training=True, eps=1e-5).numpy().reshape(x.shape)
            if relu:
                ref = np.maximum(ref, 0.0)
            _close(out, ref, 1e-12, f"batch_norm {(N, C, H, W)} relu={relu}")
            xs = np.transpose(x, (1, 2, 0, 3, 4)).reshape(4, C, -1)
            _close(mean, xs.mean(axis=2), 1e-13, "mean")
            _close(var, xs.var(axis=2, ddof=0), 1e-13, "biased var")


def pin_iqbn_moments(orc):
    """After IQBN each (component, channel) has mean beta and biased variance
    gamma^2 sigma^2 / (sigma^2 + eps); gamma = 1, beta = 0 gives mean 0, var ~ 1."""
    rng = _rng(24)
    N, C, H, W = 3, 4, 5, 7
    x = rng.standard_normal((N, 4, C, H, W)) * 2.0 + 5.0
    g = rng.uniform(0.5, 1.5, (4, C))
    b = rng.standard_normal((4, C))
    eps = 1e-3
    out, mean, var = orc.iqbn(x, g, b, eps)
    os_ = np.transpose(out, (1, 2, 0, 3, 4)).reshape(4, C, -1)
    _close(os_.mean(axis=2), b, 1e-12, "output mean = beta")
    _close(os_.var(axis=2), g * g * var / (var + eps), 1e-12, "output variance")
    out1, _, _ = orc.iqbn(x, np.ones((4, C)), np.zeros((4, C)), 1e-12)
    o1 = np.transpose(out1, (1, 2, 0, 3, 4)).reshape(4, C, -1)
    _close(o1.mean(axis=2), np.zeros((4, C)), 1e-12, "unit mean")
    _close(o1.var(axis=2), np.ones((4, C)), 1e-9, "unit var")


def pin_iqbn_degenerate(orc):
    """One sample per channel, or a constant channel: variance 0, output beta."""
    rng = _rng(25)
    g = rng.uniform(0.5, 1.5, (4, 2))
    b = rng.standard_normal((4, 2))
    x = rng.standard_normal((1, 4, 2, 1, 1))
    out, mean, var = orc.iqbn(x, g, b, 1e-5)
    _close(var, np.zeros((4, 2)), 0, "n=1 var")
    _close(out.reshape(4, 2), b, 1e-15, "n=1 out")
    xc = np.full((2, 4, 2, 3, 3), 2.5)
    out, mean, var = orc.iqbn(xc, g, b, 1e-5)
    _close(mean, np.full((4, 2), 2.5), 0, "const mean")
    _close(out, np.broadcast_to(b[None, :, :, None, None], out.shape), 1e-15, "const out")


# ---------------------------- separable convolution ---------------------------

def eq7_signs():
    """S[p, q] of the eq. 7 fixture; raises if a term convolves W_a with x_b
    for a != b (eq. 7 has none)."""
    S = np.zeros((4, 4))
    for ln in _lines("separable_eq7.txt"):
        head, terms = ln.split(":")
        p = COMP[head.strip()]
        for t in terms.split():
            sign = -1.0 if t[0] == "-" else 1.0
            wpart, xpart = t[1:].split("*")
            a, b = COMP[wpart.split("_")[1]], COMP[xpart.split("_")[1]]
            assert a == b, "eq. 7 fixture: cross term"
            S[p, a] += sign
    return S


def eq9_mixing():
    """The mixing matrix M printed for the backward pass (eq. 9 fixture)."""
    return np.array([[float(v) for v in ln.split()] for ln in _lines("mixing_matrix_eq9.txt")])


def _sep_unit(orc, a, b):
    x = np.eye(4)[b].reshape(1, 4, 1, 1, 1)
    w = np.eye(4)[a].reshape(4, 1, 1, 1, 1)
    return orc.qconv2d_separable(x, w).reshape(4)


def pin_separable_eq7_terms(orc):
    """W = e_a, X = e_b gives S[:, a] of eq. 7 when a == b and zero otherwise
    (no cross-component terms)."""
    S = eq7_signs()
    for a in range(4):
        for b in range(4):
            ref = S[:, a] if a == b else np.zeros(4)
            _close(_sep_unit(orc, a, b), ref, 0, f"eq. 7 W_{a} x_{b}")


def pin_separable_mixing_transpose(orc):
    """The sign matrix the oracle applies is the transpose of the printed
    backward mixing matrix M (eq. 9), and S S^T = 4 I."""
    S = np.stack([_sep_unit(orc, q, q) for q in range(4)], axis=1)
    _close(S, eq9_mixing().T, 0, "S = M^T")
    _close(S @ S.T, 4.0 * np.eye(4), 0, "S S^T = 4 I")


def pin_separable_real_row(orc):
    """Row r of eq. 7 is exactly row r of the Hamilton product (eq. 5): the
    separable and the full convolution agree on the real component."""
    rng = _rng(30)
    for (N, Cin, Cout, H, W, k, s, p, d) in CONV_SWEEP[:4]:
        x = rng.standard_normal((N, 4, Cin, H, W))
        w = rng.standard_normal((4, Cout, Cin, k, k))
        b = rng.standard_normal((4, Cout))
        _close(orc.qconv2d_separable(x, w, b, s, p, d)[:, 0], orc.qconv2d(x, w, b, s, p, d)[:, 0],
               1e-12, "separable row r")


def pin_separable_block_matrix(orc):
    """Agreement with torch's fp64 conv2d of the real 4Cin -> 4Cout weight
    whose block (p, q) is S[p, q] * W_q (eq. 7 fixture), with bias."""
    S = eq7_signs()
    rng = _rng(31)
    for (N, Cin, Cout, H, W, k, s, p, d) in CONV_SWEEP:
        x = rng.standard_normal((N, 4, Cin, H, W))
        w = rng.standard_normal((4, Cout, Cin, k, k))
        b = rng.standard_normal((4, Cout))
        wb = np.concatenate([np.concatenate([S[pp, q] * w[q] for q in range(4)], axis=1)
                             for pp in range(4)], axis=0)
        ref = F.conv2d(torch.from_numpy(np.ascontiguousarray(x.reshape(N, 4 * Cin, H, W))),
                       torch.from_numpy(wb), torch.from_numpy(b.reshape(-1)),
                       stride=s, padding=p, dilation=d).numpy()
        y = orc.qconv2d_separable(x, w, b, s, p, d)
        _close(y, ref.reshape(y.shape), 1e-12, f"separable block {(N, Cin, Cout, H, W, k, s, p, d)}")


# ------------------------------- conv gradients -------------------------------

def pin_backward_adjoint(orc):
    """The forward pass is linear in X and in W, so <conv(X; W), G> equals
    <X, dX> and <W, dW> for the oracle's gradients at dL/dY = G; and dbias is
    G summed over batch and pixels."""
    rng = _rng(32)
    for (N, Cin, Cout, H, W, k, s, p, d) in CONV_SWEEP:
        x = rng.standard_normal((N, 4, Cin, H, W))
        w = rng.standard_normal((4, Cout, Cin, k, k))
        y = orc.qconv2d(x, w, None, s, p, d)
        g = rng.standard_normal(y.shape)
        dx, dw, db = orc.qconv2d_backward(x, w, g, s, p, d)
        lhs = float(np.sum(y * g))
        tag = str((N, Cin, Cout, H, W, k, s, p, d))
        _close(np.sum(x * dx), lhs, 1e-12, f"<X, dX> {tag}")
        _close(np.sum(w * dw), lhs, 1e-12, f"<W, dW> {tag}")
        _close(db, g.sum(axis=(0, 3, 4)), 1e-13, f"dbias {tag}")


def pin_backward_autograd(orc):
    """Gradients equal torch autograd (fp64) through conv2d of the eq. 6 block
    weight assembled from W_r..W_k."""
    sign, comp = eq6_matrix_pattern()
    rng = _rng(33)
    for (N, Cin, Cout, H, W, k, s, p, d) in CONV_SWEEP:
        x = rng.standard_normal((N, 4, Cin, H, W))
        w = rng.standard_normal((4, Cout, Cin, k, k))
        b = rng.standard_normal((4, Cout))
        xt = torch.from_numpy(x.reshape(N, 4 * Cin, H, W).copy()).requires_grad_(True)
        wt = torch.from_numpy(w.copy()).requires_grad_(True)
        bt = torch.from_numpy(b.copy()).requires_grad_(True)
        wb = torch.cat([torch.cat([float(sign[pp, q]) * wt[comp[pp, q]] for q in range(4)], dim=1)
                        for pp in range(4)], dim=0)
        y = F.conv2d(xt, wb, bt.reshape(-1), stride=s, padding=p, dilation=d)
        g = rng.standard_normal(tuple(y.shape))
        y.backward(torch.from_numpy(g))
        dx, dw, db = orc.qconv2d_backward(x, w, g.reshape(N, 4, Cout, y.shape[2], y.shape[3]), s, p, d)
        tag = str((N, Cin, Cout, H, W, k, s, p, d))
        _close(dx, xt.grad.numpy().reshape(x.shape), 1e-12, f"autograd dX {tag}")
        _close(dw, wt.grad.numpy(), 1e-12, f"autograd dW {tag}")
        _close(db, bt.grad.numpy(), 1e-12, f"autograd dbias {tag}")


def pin_backward_conjugate_kernel(orc):
    """For stride 1, dX is the forward convolution of dY with the kernel
    transposed (Cin <-> Cout), flipped in space and conjugated
    (w_r, -w_i, -w_j, -w_k), padded by d(k-1) - p: L(w)^T = L(conj w)."""
    rng = _rng(34)
    for (N, Cin, Cout, H, W, k, p, d) in [(2, 3, 2, 7, 6, 3, 1, 1), (1, 2, 3, 8, 9, 5, 2, 1),
                                          (1, 2, 2, 9, 8, 3, 2, 2), (2, 3, 4, 5, 5, 1, 0, 1)]:
        x = rng.standard_normal((N, 4, Cin, H, W))
        w = rng.standard_normal((4, Cout, Cin, k, k))
        g = rng.standard_normal(orc.qconv2d(x, w, None, 1, p, d).shape)
        dx, _, _ = orc.qconv2d_backward(x, w, g, 1, p, d)
        wt = np.transpose(w, (0, 2, 1, 3, 4))[:, :, :, ::-1, ::-1] * np.array([1, -1, -1, -1])[:, None, None, None, None]
        _close(dx, orc.qconv2d(g, wt, None, 1, d * (k - 1) - p, d), 1e-12, f"conjugate kernel {(k, p, d)}")


# --------------------------------- IQBN extras ---------------------------------

def pin_iqbn_inference_batch_norm(orc):
    """Inference IQBN equals torch's fp64 batch_norm with running statistics
    (training=False), with and without ReLU."""
    rng = _rng(35)
    N, C, H, W = 3, 4, 5, 6
    x = rng.standard_normal((N, 4, C, H, W)) * 2.0 + 1.0
    m = rng.standard_normal((4, C))
    v = rng.uniform(0.2, 3.0, (4, C))
    g = rng.uniform(0.5, 1.5, (4, C))
    b = rng.standard_normal((4, C))
    for relu in (False, True):
        out = orc.iqbn_inference(x, m, v, g, b, 1e-3, relu)
        ref = F.batch_norm(torch.from_numpy(x.reshape(N, 4 * C, H, W)), torch.from_numpy(m.reshape(-1)),
                           torch.from_numpy(v.reshape(-1)), torch.from_numpy(g.reshape(-1)),
                           torch.from_numpy(b.reshape(-1)), training=False, eps=1e-3).numpy()
        if relu:
            ref = np.maximum(ref, 0.0)
        _close(out, ref.reshape(x.shape), 1e-12, f"inference batch_norm relu={relu}")


def pin_iqbn_inference_batch_stats(orc):
    """With the batch's own mean and biased variance as the stored
    statistics, inference IQBN reproduces training-mode IQBN."""
    rng = _rng(36)
    x = rng.standard_normal((2, 4, 3, 4, 5)) * 1.5 - 0.5
    g = rng.uniform(0.5, 1.5, (4, 3))
    b = rng.standard_normal((4, 3))
    out, mean, var = orc.iqbn(x, g, b, 1e-5, True)
    _close(orc.iqbn_inference(x, mean, var, g, b, 1e-5, True), out, 1e-13, "inference = training")


def pin_iqbn_backward_autograd(orc):
    """IQBN gradients equal torch autograd (fp64) through training-mode
    batch_norm over the 4C real channels, with and without ReLU."""
    rng = _rng(37)
    for (N, C, H, W) in [(3, 2, 4, 5), (2, 3, 3, 3), (1, 1, 1, 6)]:
        x = rng.standard_normal((N, 4, C, H, W)) * 2.0 + rng.standard_normal((1, 4, C, 1, 1))
        g = rng.uniform(0.5, 1.5, (4, C))
        b = rng.standard_normal((4, C))
        dout = rng.standard_normal(x.shape)
        for relu in (False, True):
            xt = torch.from_numpy(x.reshape(N, 4 * C, H, W).copy()).requires_grad_(True)
            gt = torch.from_numpy(g.reshape(-1).copy()).requires_grad_(True)
            bt = torch.from_numpy(b.reshape(-1).copy()).requires_grad_(True)
            y = F.batch_norm(xt, None, None, gt, bt, training=True, eps=1e-5)
            if relu:
                y = torch.relu(y)
            y.backward(torch.from_numpy(dout.reshape(N, 4 * C, H, W)))
            dx, dg, db = orc.iqbn_backward(x, g, b, dout, 1e-5, relu)
            tag = f"{(N, C, H, W)} relu={relu}"
            _close(dx, xt.grad.numpy().reshape(x.shape), 1e-11, f"iqbn dX {tag}")
            _close(dg, gt.grad.numpy().reshape(4, C), 1e-11, f"iqbn dgamma {tag}")
            _close(db, bt.grad.numpy().reshape(4, C), 1e-11, f"iqbn dbeta {tag}")


def pin_iqbn_backward_zero_sum(orc):
    """Without ReLU the input gradient of each (component, channel) sums to
    zero: shifting a channel's inputs by a constant leaves the output alone."""
    rng = _rng(38)
    x = rng.standard_normal((3, 4, 2, 4, 4)) + 3.0
    dx, _, _ = orc.iqbn_backward(x, rng.uniform(0.5, 1.5, (4, 2)), rng.standard_normal((4, 2)),
                                 rng.standard_normal(x.shape), 1e-5, False)
    _close(dx.sum(axis=(0, 3, 4)), np.zeros((4, 2)), 1e-12, "sum dX")


# ----------------------------- Poincare mapping -----------------------------

def pin_poincare_unit_norm(orc):
    """Eq. 4 lands on the unit sphere: ((1-n^2)^2 + 4n^2) = (1+n^2)^2."""
    rng = _rng(39)
    rgb = np.concatenate([rng.uniform(0, 1, (2, 3, 5, 4)), rng.standard_normal((1, 3, 5, 4)) * 10], axis=0)
    q = orc.poincare(rgb)
    _close(np.linalg.norm(q[:, :, 0], axis=1), np.ones((3, 5, 4)), 1e-14, "unit norm")


def pin_poincare_inverse(orc):
    """The inverse stereographic projection (q_i, q_j, q_k) / (1 + q_r)
    recovers (r, g, b) in order."""
    rng = _rng(40)
    rgb = rng.uniform(0, 1, (2, 3, 6, 5))
    q = orc.poincare(rgb)[:, :, 0]
    _close(q[:, 1:] / (1.0 + q[:, :1]), rgb, 1e-14, "inverse")


def pin_poincare_special_points(orc):
    """Black maps to 1; the unit colour axes map to i, j and k."""
    rgb = np.zeros((1, 3, 1, 4))
    rgb[0, 0, 0, 1] = rgb[0, 1, 0, 2] = rgb[0, 2, 0, 3] = 1.0
    q = orc.poincare(rgb)[0, :, 0, 0, :].T
    _close(q, np.array([UNIT["1"], UNIT["i"], UNIT["j"], UNIT["k"]]), 0, "special points")


# --------------------------- separable conv gradients --------------------------

def pin_separable_backward_adjoint(orc):
    """eq. 7 is linear in x and in W: <sep(x; W), G> = <x, dx> = <W, dW> for
    the oracle's gradients at dL/dY = G; dbias is G summed."""
    rng = _rng(35)
    for (N, Cin, Cout, H, W, k, s, p, d) in CONV_SWEEP:
        x = rng.standard_normal((N, 4, Cin, H, W))
        w = rng.standard_normal((4, Cout, Cin, k, k))
        y = orc.qconv2d_separable(x, w, None, s, p, d)
        g = rng.standard_normal(y.shape)
        dx, dw, db = orc.qconv2d_separable_backward(x, w, g, s, p, d)
        lhs = float(np.sum(y * g))
        tag = str((N, Cin, Cout, H, W, k, s, p, d))
        _close(np.sum(x * dx), lhs, 1e-12, f"separable <X, dX> {tag}")
        _close(np.sum(w * dw), lhs, 1e-12, f"separable <W, dW> {tag}")
        _close(db, g.sum(axis=(0, 3, 4)), 1e-13, f"separable dbias {tag}")


def pin_separable_backward_autograd(orc):
    """Gradients equal torch autograd (fp64) through conv2d of the real block
    weight whose block (p, q) is S[p, q] * W_q, S from the eq. 7 fixture."""
    S = eq7_signs()
    rng = _rng(36)
    for (N, Cin, Cout, H, W, k, s, p, d) in CONV_SWEEP:
        x = rng.standard_normal((N, 4, Cin, H, W))
        w = rng.standard_normal((4, Cout, Cin, k, k))
        b = rng.standard_normal((4, Cout))
        xt = torch.from_numpy(x.reshape(N, 4 * Cin, H, W).copy()).requires_grad_(True)
        wt = torch.from_numpy(w.copy()).requires_grad_(True)
        bt = torch.from_numpy(b.copy()).requires_grad_(True)
        wb = torch.cat([torch.cat([float(S[pp, q]) * wt[q] for q in range(4)], dim=1) for pp in range(4)], dim=0)
        y = F.conv2d(xt, wb, bt.reshape(-1), stride=s, padding=p, dilation=d)
        g = rng.standard_normal(tuple(y.shape))
        y.backward(torch.from_numpy(g))
        dx, dw, db = orc.qconv2d_separable_backward(x, w, g.reshape(N, 4, Cout, y.shape[2], y.shape[3]), s, p, d)
        tag = str((N, Cin, Cout, H, W, k, s, p, d))
        _close(dx, xt.grad.numpy().reshape(x.shape), 1e-12, f"separable autograd dX {tag}")
        _close(dw, wt.grad.numpy(), 1e-12, f"separable autograd dW {tag}")
        _close(db, bt.grad.numpy(), 1e-12, f"separable autograd dbias {tag}")


def pin_separable_backward_mixing(orc):
    """With every W_q = 1 (one 1x1 channel) the input gradient of component q
    is sum_p M[q][p] dY_p: probing with unit output gradients reproduces the
    printed matrix M of eq. 9 column by column, and the weight gradient of
    W_q for x = e_q is that same mixed component."""
    M = eq9_mixing()
    w = np.ones((4, 1, 1, 1, 1))
    got_x, got_w = np.zeros((4, 4)), np.zeros((4, 4))
    for pp in range(4):
        g = np.eye(4)[pp].reshape(1, 4, 1, 1, 1)
        dx, _, _ = orc.qconv2d_separable_backward(np.zeros((1, 4, 1, 1, 1)), w, g)
        got_x[:, pp] = dx.reshape(4)
        for q in range(4):
            _, dw, _ = orc.qconv2d_separable_backward(np.eye(4)[q].reshape(1, 4, 1, 1, 1), w, g)
            got_w[q, pp] = dw.reshape(4)[q]
    _close(got_x, M, 0, "dX mixing = M (eq. 9)")
    _close(got_w, M, 0, "dW mixing = M (eq. 9)")


ALL_PINS = [
    pin_eq2_unit_relations, pin_unit_table_derived, pin_complex_model, pin_eq6_matrix,
    pin_eq5_expansion, pin_orientation, pin_identity_kernel, pin_norm, pin_conjugate_adjoint,
    pin_real_reduction, pin_complex_reduction, pin_block_matrix, pin_brute_force_complex_model,
    pin_associativity, pin_linearity, pin_bias,
    pin_iqbn_batch_norm, pin_iqbn_moments, pin_iqbn_degenerate,
    pin_separable_eq7_terms, pin_separable_mixing_transpose, pin_separable_real_row,
    pin_separable_block_matrix,
    pin_backward_adjoint, pin_backward_autograd, pin_backward_conjugate_kernel,
    pin_separable_backward_adjoint, pin_separable_backward_autograd, pin_separable_backward_mixing,
    pin_iqbn_inference_batch_norm, pin_iqbn_inference_batch_stats,
    pin_iqbn_backward_autograd, pin_iqbn_backward_zero_sum,
    pin_poincare_unit_norm, pin_poincare_inverse, pin_poincare_special_points,
]
