"""CPU oracle for the QUAN hot path -- test infrastructure only.

Slow, plain fp64 reference implementations, written from the paper in C
(quan_oracle.c): the quaternion convolution (Section III-B, eqs. 5/6) and its
gradients, the separable convolution (eq. 7) and its gradients (eqs. 8-10), Independent Quaternion Batch
Normalization (Section III-C, eqs. 11/12) in training and inference form and
its gradients, and the Poincare input mapping (Section III-A, eq. 4).
Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this package; the GPU library never calls it and shares no code with it.

All arrays use the paper's logical layout: activations [N, 4, C, H, W] with the
quaternion component axis q in {r, i, j, k}, weights as four real kernels
[4, Cout, Cin, kh, kw], bias [4, Cout], IQBN parameters [4, C].
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")

_D = ctypes.POINTER(ctypes.c_double)
_I64 = ctypes.c_int64


def _f64(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a):
    return a.ctypes.data_as(_D) if a is not None else None


def _pair(v):
    return (int(v), int(v)) if np.isscalar(v) else (int(v[0]), int(v[1]))


class Oracle:
    """ctypes front end of one build of quan_oracle.c."""

    def __init__(self, lib_path=LIB_PATH):
        lib = ctypes.CDLL(lib_path)
        lib.quan_oracle_hamilton.argtypes = [_D, _D, _D]
        lib.quan_oracle_hamilton.restype = None
        lib.quan_oracle_out_size.argtypes = [_I64] * 5
        lib.quan_oracle_out_size.restype = _I64
        lib.quan_oracle_qconv2d.argtypes = [_D, _D, _D, _D] + [_I64] * 13
        lib.quan_oracle_qconv2d.restype = None
        lib.quan_oracle_iqbn.argtypes = [_D, _D, _D, ctypes.c_double, ctypes.c_int,
                                         _D, _D, _D] + [_I64] * 4
        lib.quan_oracle_iqbn.restype = None
        lib.quan_oracle_qconv2d_separable.argtypes = [_D, _D, _D, _D] + [_I64] * 13
        lib.quan_oracle_qconv2d_separable.restype = None
        lib.quan_oracle_iqbn_inference.argtypes = [_D, _D, _D, _D, _D, ctypes.c_double, ctypes.c_int,
                                                   _D] + [_I64] * 4
        lib.quan_oracle_iqbn_inference.restype = None
        lib.quan_oracle_poincare.argtypes = [_D, _D] + [_I64] * 3
        lib.quan_oracle_poincare.restype = None
        lib.quan_oracle_qconv2d_backward.argtypes = [_D] * 6 + [_I64] * 13
        lib.quan_oracle_qconv2d_backward.restype = None
        lib.quan_oracle_qconv2d_separable_backward.argtypes = [_D] * 6 + [_I64] * 13
        lib.quan_oracle_qconv2d_separable_backward.restype = None
        lib.quan_oracle_iqbn_backward.argtypes = [_D, _D, _D, ctypes.c_double, ctypes.c_int,
                                                  _D, _D, _D, _D] + [_I64] * 4
        lib.quan_oracle_iqbn_backward.restype = None
        self.lib = lib
        self.path = lib_path

    def hamilton(self, p, q):
        """Hamilton product p (x) q of two quaternions (r, i, j, k), eq. 3."""
        p, q = _f64(p), _f64(q)
        assert p.shape == (4,) and q.shape == (4,)
        out = np.empty(4)
        self.lib.quan_oracle_hamilton(_ptr(p), _ptr(q), _ptr(out))
        return out

    def out_size(self, n, k, stride, pad, dil):
        return int(self.lib.quan_oracle_out_size(n, k, stride, pad, dil))

    def qconv2d(self, x, w, bias=None, stride=1, pad=0, dilation=1):
        """Quaternion convolution Y = W (x) X (eq. 5), fp64.

        x: [N, 4, Cin, H, W]; w: [4, Cout, Cin, kh, kw] (W_r, W_i, W_j, W_k);
        bias: [4, Cout] or None.  Returns y: [N, 4, Cout, Ho, Wo]."""
        x, w = _f64(x), _f64(w)
        N, four, Cin, H, W = x.shape
        assert four == 4 and w.shape[0] == 4 and w.shape[2] == Cin
        Cout, KH, KW = w.shape[1], w.shape[3], w.shape[4]
        b = None if bias is None else _f64(bias)
        if b is not None:
            assert b.shape == (4, Cout)
        sh, sw = _pair(stride)
        ph, pw = _pair(pad)
        dh, dw = _pair(dilation)
        Ho, Wo = self.out_size(H, KH, sh, ph, dh), self.out_size(W, KW, sw, pw, dw)
        if Ho <= 0 or Wo <= 0:
            raise ValueError("empty output")
        y = np.zeros((N, 4, Cout, Ho, Wo))
        self.lib.quan_oracle_qconv2d(_ptr(x), _ptr(w), _ptr(b), _ptr(y),
                                     N, Cin, H, W, Cout, KH, KW, sh, sw, ph, pw, dh, dw)
        return y

    def _conv_dims(self, x, w, stride, pad, dilation):
        N, four, Cin, H, W = x.shape
        assert four == 4 and w.shape[0] == 4 and w.shape[2] == Cin
        Cout, KH, KW = w.shape[1], w.shape[3], w.shape[4]
        sh, sw = _pair(stride)
        ph, pw = _pair(pad)
        dh, dw = _pair(dilation)
        Ho, Wo = self.out_size(H, KH, sh, ph, dh), self.out_size(W, KW, sw, pw, dw)
        if Ho <= 0 or Wo <= 0:
            raise ValueError("empty output")
        return (N, Cin, H, W, Cout, KH, KW, sh, sw, ph, pw, dh, dw), Ho, Wo

    def qconv2d_separable(self, x, w, bias=None, stride=1, pad=0, dilation=1):
        """Separable QUAN convolution (eq. 7), fp64: y_p = bias_p +
        sum_q S[p, q] (W_q (*) x_q).  Shapes as in qconv2d."""
        x, w = _f64(x), _f64(w)
        dims, Ho, Wo = self._conv_dims(x, w, stride, pad, dilation)
        b = None if bias is None else _f64(bias)
        if b is not None:
            assert b.shape == (4, dims[4])
        y = np.zeros((dims[0], 4, dims[4], Ho, Wo))
        self.lib.quan_oracle_qconv2d_separable(_ptr(x), _ptr(w), _ptr(b), _ptr(y), *dims)
        return y

    def qconv2d_backward(self, x, w, dy, stride=1, pad=0, dilation=1):
        """Gradients of qconv2d (eq. 5) for dL/dY = dy: returns (dx, dw, db)
        shaped like x, w and the bias [4, Cout]."""
        x, w, dy = _f64(x), _f64(w), _f64(dy)
        dims, Ho, Wo = self._conv_dims(x, w, stride, pad, dilation)
        assert dy.shape == (dims[0], 4, dims[4], Ho, Wo)
        dx, dwt, db = np.empty_like(x), np.empty_like(w), np.empty((4, dims[4]))
        self.lib.quan_oracle_qconv2d_backward(_ptr(x), _ptr(w), _ptr(dy), _ptr(dx), _ptr(dwt), _ptr(db),
                                              *dims)
        return dx, dwt, db

    def qconv2d_separable_backward(self, x, w, dy, stride=1, pad=0, dilation=1):
        """Gradients of qconv2d_separable (eq. 7) for dL/dY = dy, by eqs. 8-10
        with the printed mixing matrix M: returns (dx, dw, db)."""
        x, w, dy = _f64(x), _f64(w), _f64(dy)
        dims, Ho, Wo = self._conv_dims(x, w, stride, pad, dilation)
        assert dy.shape == (dims[0], 4, dims[4], Ho, Wo)
        dx, dwt, db = np.empty_like(x), np.empty_like(w), np.empty((4, dims[4]))
        self.lib.quan_oracle_qconv2d_separable_backward(_ptr(x), _ptr(w), _ptr(dy), _ptr(dx), _ptr(dwt),
                                                        _ptr(db), *dims)
        return dx, dwt, db

    def iqbn_inference(self, x, mean, var, gamma, beta, eps=1e-5, relu=False):
        """IQBN with given (running) statistics, eq. 12, fp64."""
        x = _f64(x)
        N, four, C, H, W = x.shape
        assert four == 4
        m, v = _f64(mean).reshape(4, C), _f64(var).reshape(4, C)
        g, b = _f64(gamma).reshape(4, C), _f64(beta).reshape(4, C)
        out = np.empty_like(x)
        self.lib.quan_oracle_iqbn_inference(_ptr(x), _ptr(m), _ptr(v), _ptr(g), _ptr(b), float(eps),
                                            int(bool(relu)), _ptr(out), N, C, H, W)
        return out

    def iqbn_backward(self, x, gamma, beta, dout, eps=1e-5, relu=False):
        """Gradients of training-mode IQBN (+ ReLU) for dL/dout = dout:
        returns (dx, dgamma, dbeta)."""
        x, dout = _f64(x), _f64(dout)
        N, four, C, H, W = x.shape
        assert four == 4 and dout.shape == x.shape
        g, b = _f64(gamma).reshape(4, C), _f64(beta).reshape(4, C)
        dx, dg, db = np.empty_like(x), np.empty((4, C)), np.empty((4, C))
        self.lib.quan_oracle_iqbn_backward(_ptr(x), _ptr(g), _ptr(b), float(eps), int(bool(relu)),
                                           _ptr(dout), _ptr(dx), _ptr(dg), _ptr(db), N, C, H, W)
        return dx, dg, db

    def poincare(self, rgb):
        """Poincare mapping of eq. 4: rgb [N, 3, H, W] -> q [N, 4, 1, H, W]."""
        rgb = _f64(rgb)
        N, three, H, W = rgb.shape
        assert three == 3
        q = np.empty((N, 4, 1, H, W))
        self.lib.quan_oracle_poincare(_ptr(rgb), _ptr(q), N, H, W)
        return q

    def iqbn(self, x, gamma, beta, eps=1e-5, relu=False):
        """Independent Quaternion Batch Normalization (eqs. 11/12), two-pass fp64.

        x: [N, 4, C, H, W]; gamma, beta: [4, C].  Returns (out, mean, var) with
        mean/var the per-(component, channel) batch mean and biased variance."""
        x = _f64(x)
        N, four, C, H, W = x.shape
        assert four == 4
        g, b = _f64(gamma).reshape(4, C), _f64(beta).reshape(4, C)
        out = np.empty_like(x)
        mean = np.empty((4, C))
        var = np.empty((4, C))
        self.lib.quan_oracle_iqbn(_ptr(x), _ptr(g), _ptr(b), float(eps), int(bool(relu)),
                                  _ptr(out), _ptr(mean), _ptr(var), N, C, H, W)
        return out, mean, var


_default = None


def default() -> Oracle:
    """The oracle built from oracle/quan_oracle.c (built on first use)."""
    global _default
    if _default is None:
        if not os.path.exists(LIB_PATH):
            from . import build as _b
            _b.build()
        _default = Oracle(LIB_PATH)
    return _default


def hamilton(p, q):
    return default().hamilton(p, q)


def out_size(n, k, stride, pad, dil):
    return default().out_size(n, k, stride, pad, dil)


def qconv2d(x, w, bias=None, stride=1, pad=0, dilation=1):
    return default().qconv2d(x, w, bias, stride, pad, dilation)


def iqbn(x, gamma, beta, eps=1e-5, relu=False):
    return default().iqbn(x, gamma, beta, eps, relu)


def qconv2d_separable(x, w, bias=None, stride=1, pad=0, dilation=1):
    return default().qconv2d_separable(x, w, bias, stride, pad, dilation)


def qconv2d_backward(x, w, dy, stride=1, pad=0, dilation=1):
    return default().qconv2d_backward(x, w, dy, stride, pad, dilation)


def qconv2d_separable_backward(x, w, dy, stride=1, pad=0, dilation=1):
    return default().qconv2d_separable_backward(x, w, dy, stride, pad, dilation)


def iqbn_inference(x, mean, var, gamma, beta, eps=1e-5, relu=False):
    return default().iqbn_inference(x, mean, var, gamma, beta, eps, relu)


def iqbn_backward(x, gamma, beta, dout, eps=1e-5, relu=False):
    return default().iqbn_backward(x, gamma, beta, dout, eps, relu)


def poincare(rgb):
    return default().poincare(rgb)
