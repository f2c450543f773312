"""Thin ctypes binding of libquan (include/quan.h).

Argument marshalling only: the functions here check tensor shapes, dtypes and
strides, pass raw device pointers, sizes and torch's current HIP stream to the
C ABI, and raise on a non-zero status.  Every step of the computation runs in
libquan's HIP kernels; there is no fallback.  If libquan.so is missing or
cannot be loaded, the first call raises.

Quaternion feature maps are tensors of logical shape [N, 4, C, H, W]
(component axis r, i, j, k) whose memory is channels-last by component,
[N][H][W][4][C]; ``to_device_layout`` produces that layout and ``empty_qmap``
allocates it.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libquan.so")

QUAN_F32, QUAN_BF16 = 0, 1
_STATUS = {0: "QUAN_OK", -1: "QUAN_ERR_NULL", -2: "QUAN_ERR_SHAPE", -3: "QUAN_ERR_DTYPE",
           -4: "QUAN_ERR_ALIGN", -5: "QUAN_ERR_ALIAS", -6: "QUAN_ERR_UNSUPPORTED",
           -7: "QUAN_ERR_HIP", -8: "QUAN_ERR_NOMEM", -9: "QUAN_ERR_LAYOUT"}
QUAN_ERR_LAYOUT = -9


class QuanTensor(ctypes.Structure):
    """struct quan_tensor: device pointer, dtype, and up to 5 (extent, stride
    in elements) axes."""
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("shape", ctypes.c_int64 * 5), ("strides", ctypes.c_int64 * 5)]


def describe(t):
    """A quan_tensor for a torch tensor (its real shape and strides), or None."""
    if t is None:
        return None
    if t.dim() > 5:
        raise ValueError("quan_tensor holds at most 5 axes")
    d = QuanTensor()
    d.data = t.data_ptr()
    d.dtype = _dtype_code(t)
    d.ndim = t.dim()
    for i, (n, st) in enumerate(zip(t.shape, t.stride())):
        d.shape[i] = n
        d.strides[i] = st
    return d

# Every symbol include/quan.h declares, with its ctypes signature.
_vp, _i32, _f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float
SIGNATURES = {
    "quan_qconv2d_forward": (ctypes.c_int, [_vp] * 6 + [_i32] * 6 + [_vp] + [_i32] * 8 + [_vp]),
    "quan_qconv2d_forward_desc": (ctypes.c_int, [ctypes.c_void_p] * 6 + [ctypes.POINTER(ctypes.c_int32)] * 3
                                  + [ctypes.c_void_p, _vp]),
    "quan_iqbn_forward_desc": (ctypes.c_int, [_vp] * 3 + [_f32] + [_vp] * 4),
    "quan_iqbn_relu_forward_desc": (ctypes.c_int, [_vp] * 3 + [_f32] + [_vp] * 4),
    "quan_qconv2d_packed_bytes": (ctypes.c_int64, [_i32] * 5),
    "quan_qconv2d_pack_weights": (ctypes.c_int, [_vp] * 4 + [_i32] * 5 + [_vp, ctypes.c_int64, _vp]),
    "quan_qconv2d_forward_packed": (ctypes.c_int, [_vp] * 3 + [_i32] * 6 + [_vp] + [_i32] * 8 + [_vp]),
    "quan_qconv2d_separable_forward": (ctypes.c_int, [_vp] * 6 + [_i32] * 6 + [_vp] + [_i32] * 8 + [_vp]),
    "quan_qconv2d_separable_forward_packed": (ctypes.c_int, [_vp] * 3 + [_i32] * 6 + [_vp] + [_i32] * 8
                                              + [_vp]),
    "quan_qconv2d_iqbn_forward": (ctypes.c_int, [_vp] * 3 + [_i32] * 6 + [_vp, _vp, _f32, _i32, _i32]
                                  + [_vp] * 3 + [_i32] * 8 + [_vp]),
    "quan_qconv2d_iqbn_inference": (ctypes.c_int, [_vp] * 3 + [_i32] * 6 + [_vp] * 4 + [_f32, _i32, _vp]
                                    + [_i32] * 8 + [_vp]),
    "quan_poincare_map": (ctypes.c_int, [_vp, _vp] + [_i32] * 4 + [_vp]),
    "quan_qconv2d_poincare_forward": (ctypes.c_int, [_vp] * 3 + [_i32] * 6 + [_vp] + [_i32] * 7 + [_vp]),
    "quan_qconv2d_backward_data": (ctypes.c_int, [_vp] * 5 + [_i32] * 6 + [_vp] + [_i32] * 8 + [_vp]),
    "quan_qconv2d_backward_weight": (ctypes.c_int, [_vp] * 2 + [_i32] * 6 + [_vp] * 5 + [_i32] * 8 + [_vp]),
    "quan_qconv2d_separable_backward_data": (ctypes.c_int, [_vp] * 5 + [_i32] * 6 + [_vp] + [_i32] * 8 + [_vp]),
    "quan_qconv2d_separable_backward_weight": (ctypes.c_int, [_vp] * 2 + [_i32] * 6 + [_vp] * 5 + [_i32] * 8
                                               + [_vp]),
    "quan_iqbn_backward": (ctypes.c_int, [_vp] * 6 + [_f32] + [_vp] * 3 + [_i32] * 5 + [_vp]),
    "quan_iqbn_forward": (ctypes.c_int, [_vp, _vp, _vp, _f32, _vp, _vp, _vp] + [_i32] * 5 + [_vp]),
    "quan_iqbn_relu_forward": (ctypes.c_int, [_vp, _vp, _vp, _f32, _vp, _vp, _vp] + [_i32] * 5 + [_vp]),
    "quan_iqbn_forward_noalloc": (ctypes.c_int, [_vp, _vp, _vp, _f32, _vp, _vp, _vp] + [_i32] * 5 + [_vp]),
    "quan_last_error": (ctypes.c_char_p, []),
    "quan_release": (ctypes.c_int, []),
    "quan_version": (ctypes.c_char_p, []),
}

_lib = None


class QuanError(RuntimeError):
    def __init__(self, code, message):
        super().__init__(f"{_STATUS.get(code, code)}: {message}")
        self.code = code


def load_library(path: str = LIB_PATH):
    """Load libquan.so (once) and attach the C signatures."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise RuntimeError(f"libquan.so not built ({path}); run __graft_entry__.build()")
        lib = ctypes.CDLL(path)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def _check(rc):
    if rc != 0:
        raise QuanError(rc, load_library().quan_last_error().decode())


def _dtype_code(t):
    if t.dtype == torch.bfloat16:
        return QUAN_BF16
    if t.dtype == torch.float32:
        return QUAN_F32
    raise TypeError(f"unsupported dtype {t.dtype}; expected bfloat16 or float32")


def device_strides(n, c, h, w):
    """Strides (elements) of a logical [N, 4, C, H, W] map stored [N][H][W][4][C]."""
    return (h * w * 4 * c, c, 1, w * 4 * c, 4 * c)


def is_device_layout(t: torch.Tensor) -> bool:
    if t.dim() != 5 or t.shape[1] != 4:
        return False
    n, _, c, h, w = t.shape
    want = device_strides(n, c, h, w)
    return all(st == wt or sz == 1 for st, wt, sz in zip(t.stride(), want, t.shape))


def to_device_layout(t: torch.Tensor) -> torch.Tensor:
    """Logical [N, 4, C, H, W] tensor -> same values, channels-last by component."""
    assert t.dim() == 5 and t.shape[1] == 4, "expected [N, 4, C, H, W]"
    return t.permute(0, 3, 4, 1, 2).contiguous().permute(0, 3, 4, 1, 2)


def empty_qmap(n, c, h, w, dtype, device):
    return torch.empty((n, h, w, 4, c), dtype=dtype, device=device).permute(0, 3, 4, 1, 2)


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _pair(v):
    return (int(v), int(v)) if isinstance(v, int) else (int(v[0]), int(v[1]))


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def conv_out_size(n, k, stride, pad, dil):
    return (n + 2 * pad - dil * (k - 1) - 1) // stride + 1


def _ref(d):
    return ctypes.byref(d) if d is not None else None


def quan_qconv2d_forward(x, w_r, w_i, w_j, w_k, bias=None, stride=1, pad=0, dilation=1, out=None):
    """Quaternion convolution Y = W (x) X + b (Section III-B, eqs. 5/6).

    x: [N, 4, Cin, H, W] in device layout; w_*: [Cout, Cin, kh, kw] contiguous;
    bias: [4, Cout] or None.  Returns out [N, 4, Cout, Ho, Wo] (device layout).
    The tensors go to the library as descriptors with their real strides: the
    library checks shapes, dtypes and layouts (QuanError QUAN_ERR_LAYOUT for
    a map that is not channels-last by component)."""
    lib = load_library()
    if x.dim() != 5 or w_r.dim() != 4:
        raise ValueError("x must be [N, 4, Cin, H, W] and w_r [Cout, Cin, kh, kw]")
    for t in (w_r, w_i, w_j, w_k, bias, out):
        if t is not None and t.device != x.device:
            raise ValueError("all tensors must be on x's device")
    n, _, _, h, w = x.shape
    c_out, _, k_h, k_w = w_r.shape
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    dh, dw = _pair(dilation)
    if out is None:
        ho, wo = conv_out_size(h, k_h, sh, ph, dh), conv_out_size(w, k_w, sw, pw, dw)
        out = empty_qmap(n, c_out, max(ho, 1), max(wo, 1), x.dtype, x.device)
    pair = ctypes.c_int32 * 2
    descs = [describe(t) for t in (x, w_r, w_i, w_j, w_k, bias, out)]
    with torch.cuda.device(x.device):
        rc = lib.quan_qconv2d_forward_desc(*[_ref(d) for d in descs[:6]], pair(sh, sw), pair(ph, pw),
                                           pair(dh, dw), _ref(descs[6]), _stream(x.device))
    _check(rc)
    return out


def quan_qconv2d_separable_forward(x, w_r, w_i, w_j, w_k, bias=None, stride=1, pad=0, dilation=1,
                                   out=None):
    """Separable QUAN convolution (Section III-B, eq. 7): y_p = sum_q
    S[p, q] (W_q (*) x_q) + b_p.  Arguments as in quan_qconv2d_forward."""
    return _conv("quan_qconv2d_separable_forward", x, w_r, w_i, w_j, w_k, bias, stride, pad, dilation,
                 out)


def _conv(fn_name, x, w_r, w_i, w_j, w_k, bias, stride, pad, dilation, out):
    lib = load_library()
    if not is_device_layout(x):
        raise ValueError("x must be [N, 4, Cin, H, W] stored channels-last by component")
    n, _, c_in, h, w = x.shape
    for t in (w_r, w_i, w_j, w_k):
        if t.dim() != 4 or not t.is_contiguous() or t.shape[1] != c_in or t.shape != w_r.shape:
            raise ValueError("w_r..w_k must be contiguous [Cout, Cin, kh, kw] of equal shape")
        if t.dtype != x.dtype or t.device != x.device:
            raise ValueError("weights must match x in dtype and device")
    c_out, _, k_h, k_w = w_r.shape
    if bias is not None and (tuple(bias.shape) != (4, c_out) or not bias.is_contiguous()
                             or bias.dtype != x.dtype or bias.device != x.device):
        raise ValueError("bias must be a contiguous [4, Cout] tensor like x")
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    dh, dw = _pair(dilation)
    ho, wo = conv_out_size(h, k_h, sh, ph, dh), conv_out_size(w, k_w, sw, pw, dw)
    if out is None:
        out = empty_qmap(n, c_out, max(ho, 1), max(wo, 1), x.dtype, x.device)
    elif not is_device_layout(out) or tuple(out.shape) != (n, 4, c_out, ho, wo) or out.dtype != x.dtype:
        raise ValueError("out must be [N, 4, Cout, Ho, Wo] in device layout with x's dtype")
    with torch.cuda.device(x.device):
        rc = getattr(lib, fn_name)(_ptr(x), _ptr(w_r), _ptr(w_i), _ptr(w_j), _ptr(w_k),
                                   _ptr(bias), sh, sw, ph, pw, dh, dw, _ptr(out),
                                   n, c_in, h, w, c_out, k_h, k_w, _dtype_code(x),
                                   _stream(x.device))
    _check(rc)
    return out


def quan_qconv2d_packed_bytes(c_in, c_out, k_h, k_w, dtype=torch.bfloat16):
    """Bytes of packed weights for these sizes (see quan_qconv2d_pack_weights)."""
    code = QUAN_BF16 if dtype == torch.bfloat16 else QUAN_F32
    n = load_library().quan_qconv2d_packed_bytes(c_in, c_out, k_h, k_w, code)
    if n < 0:
        _check(int(n))
    return int(n)


def _check_weights(ws, like):
    w_r = ws[0]
    for t in ws:
        if t.dim() != 4 or not t.is_contiguous() or t.shape != w_r.shape:
            raise ValueError("w_r..w_k must be contiguous [Cout, Cin, kh, kw] of equal shape")
        if t.dtype != like.dtype or t.device != like.device:
            raise ValueError("weights must match in dtype and device")
    return tuple(w_r.shape)


def quan_qconv2d_pack_weights(w_r, w_i, w_j, w_k, packed=None):
    """Pack the four real kernels once for quan_qconv2d_forward_packed.

    Returns the packed buffer (a uint8 device tensor)."""
    lib = load_library()
    c_out, c_in, k_h, k_w = _check_weights((w_r, w_i, w_j, w_k), w_r)
    need = quan_qconv2d_packed_bytes(c_in, c_out, k_h, k_w, w_r.dtype)
    if packed is None:
        packed = torch.empty(need, dtype=torch.uint8, device=w_r.device)
    elif packed.numel() * packed.element_size() < need or not packed.is_contiguous():
        raise ValueError(f"packed must be a contiguous buffer of at least {need} bytes")
    with torch.cuda.device(w_r.device):
        rc = lib.quan_qconv2d_pack_weights(_ptr(w_r), _ptr(w_i), _ptr(w_j), _ptr(w_k), c_in, c_out,
                                           k_h, k_w, _dtype_code(w_r), _ptr(packed),
                                           packed.numel() * packed.element_size(),
                                           _stream(w_r.device))
    _check(rc)
    return packed


def quan_qconv2d_forward_packed(x, packed, weight_shape, bias=None, stride=1, pad=0, dilation=1,
                                out=None):
    """quan_qconv2d_forward on weights packed by quan_qconv2d_pack_weights.

    weight_shape: (Cout, Cin, kh, kw) of the kernels that were packed."""
    return _conv_packed("quan_qconv2d_forward_packed", x, packed, weight_shape, bias, stride, pad,
                        dilation, out)


def quan_qconv2d_separable_forward_packed(x, packed, weight_shape, bias=None, stride=1, pad=0,
                                          dilation=1, out=None):
    """quan_qconv2d_separable_forward on weights packed by
    quan_qconv2d_pack_weights (the same packed layout as the Hamilton conv)."""
    return _conv_packed("quan_qconv2d_separable_forward_packed", x, packed, weight_shape, bias, stride,
                        pad, dilation, out)


def _conv_packed(fn_name, x, packed, weight_shape, bias, stride, pad, dilation, out):
    lib = load_library()
    if not is_device_layout(x):
        raise ValueError("x must be [N, 4, Cin, H, W] stored channels-last by component")
    n, _, c_in, h, w = x.shape
    c_out, c_in_w, k_h, k_w = (int(v) for v in weight_shape)
    if c_in_w != c_in:
        raise ValueError("weight_shape does not match x's channels")
    if bias is not None and (tuple(bias.shape) != (4, c_out) or not bias.is_contiguous()
                             or bias.dtype != x.dtype or bias.device != x.device):
        raise ValueError("bias must be a contiguous [4, Cout] tensor like x")
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    dh, dw = _pair(dilation)
    ho, wo = conv_out_size(h, k_h, sh, ph, dh), conv_out_size(w, k_w, sw, pw, dw)
    if out is None:
        out = empty_qmap(n, c_out, max(ho, 1), max(wo, 1), x.dtype, x.device)
    elif not is_device_layout(out) or tuple(out.shape) != (n, 4, c_out, ho, wo) or out.dtype != x.dtype:
        raise ValueError("out must be [N, 4, Cout, Ho, Wo] in device layout with x's dtype")
    with torch.cuda.device(x.device):
        rc = getattr(lib, fn_name)(_ptr(x), _ptr(packed), _ptr(bias), sh, sw, ph, pw,
                                   dh, dw, _ptr(out), n, c_in, h, w, c_out, k_h, k_w,
                                   _dtype_code(x), _stream(x.device))
    _check(rc)
    return out


STATS_MODES = {"auto": 0, "epilogue": 1, "pass": 2}


def quan_qconv2d_iqbn_forward(x, packed, weight_shape, gamma, beta, bias=None, stride=1, pad=0,
                              dilation=1, eps=1e-5, relu=False, out=None, mean=None, var=None,
                              stats="auto"):
    """The convolution on packed weights followed by IQBN (+ ReLU) of its
    output.  stats: "epilogue" (per-tile statistics in the convolution's
    epilogue), "pass" (a separate statistics pass) or "auto" (the library's
    choice).  Returns (out, mean, var)."""
    lib = load_library()
    if stats not in STATS_MODES:
        raise ValueError(f"stats must be one of {sorted(STATS_MODES)}")
    if not is_device_layout(x):
        raise ValueError("x must be [N, 4, Cin, H, W] stored channels-last by component")
    n, _, c_in, h, w = x.shape
    c_out, c_in_w, k_h, k_w = (int(v) for v in weight_shape)
    if c_in_w != c_in:
        raise ValueError("weight_shape does not match x's channels")
    if bias is not None and (tuple(bias.shape) != (4, c_out) or not bias.is_contiguous()
                             or bias.dtype != x.dtype or bias.device != x.device):
        raise ValueError("bias must be a contiguous [4, Cout] tensor like x")
    for name, t in (("gamma", gamma), ("beta", beta)):
        if tuple(t.shape) != (4, c_out) or t.dtype != torch.float32 or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous float32 [4, Cout] tensor")
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    dh, dw = _pair(dilation)
    ho, wo = conv_out_size(h, k_h, sh, ph, dh), conv_out_size(w, k_w, sw, pw, dw)
    if out is None:
        out = empty_qmap(n, c_out, max(ho, 1), max(wo, 1), x.dtype, x.device)
    elif not is_device_layout(out) or tuple(out.shape) != (n, 4, c_out, ho, wo) or out.dtype != x.dtype:
        raise ValueError("out must be [N, 4, Cout, Ho, Wo] in device layout with x's dtype")
    if mean is None:
        mean = torch.empty(4, c_out, dtype=torch.float32, device=x.device)
    if var is None:
        var = torch.empty(4, c_out, dtype=torch.float32, device=x.device)
    with torch.cuda.device(x.device):
        rc = lib.quan_qconv2d_iqbn_forward(_ptr(x), _ptr(packed), _ptr(bias), sh, sw, ph, pw, dh, dw,
                                           _ptr(gamma), _ptr(beta), float(eps), int(bool(relu)),
                                           STATS_MODES[stats], _ptr(out), _ptr(mean), _ptr(var), n,
                                           c_in, h, w, c_out,
                                           k_h, k_w, _dtype_code(x), _stream(x.device))
    _check(rc)
    return out, mean, var


def quan_qconv2d_iqbn_inference(x, packed, weight_shape, running_mean, running_var, gamma, beta,
                                bias=None, stride=1, pad=0, dilation=1, eps=1e-5, relu=False, out=None):
    """Inference-mode convolution + IQBN (+ ReLU) with stored statistics,
    folded into the convolution's epilogue.  Returns out."""
    lib = load_library()
    if not is_device_layout(x):
        raise ValueError("x must be [N, 4, Cin, H, W] stored channels-last by component")
    n, _, c_in, h, w = x.shape
    c_out, c_in_w, k_h, k_w = (int(v) for v in weight_shape)
    if c_in_w != c_in:
        raise ValueError("weight_shape does not match x's channels")
    if bias is not None and (tuple(bias.shape) != (4, c_out) or not bias.is_contiguous()
                             or bias.dtype != x.dtype or bias.device != x.device):
        raise ValueError("bias must be a contiguous [4, Cout] tensor like x")
    for name, t in (("running_mean", running_mean), ("running_var", running_var), ("gamma", gamma),
                    ("beta", beta)):
        if tuple(t.shape) != (4, c_out) or t.dtype != torch.float32 or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous float32 [4, Cout] tensor")
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    dh, dw = _pair(dilation)
    ho, wo = conv_out_size(h, k_h, sh, ph, dh), conv_out_size(w, k_w, sw, pw, dw)
    if out is None:
        out = empty_qmap(n, c_out, max(ho, 1), max(wo, 1), x.dtype, x.device)
    elif not is_device_layout(out) or tuple(out.shape) != (n, 4, c_out, ho, wo) or out.dtype != x.dtype:
        raise ValueError("out must be [N, 4, Cout, Ho, Wo] in device layout with x's dtype")
    with torch.cuda.device(x.device):
        rc = lib.quan_qconv2d_iqbn_inference(_ptr(x), _ptr(packed), _ptr(bias), sh, sw, ph, pw, dh, dw,
                                             _ptr(running_mean), _ptr(running_var), _ptr(gamma),
                                             _ptr(beta), float(eps), int(bool(relu)), _ptr(out), n, c_in,
                                             h, w, c_out, k_h, k_w, _dtype_code(x), _stream(x.device))
    _check(rc)
    return out


def quan_poincare_map(rgb, out=None):
    """Poincare mapping (eq. 4) of RGB images [N, 3, H, W] (contiguous) into a
    one-channel quaternion map [N, 4, 1, H, W] in device layout."""
    lib = load_library()
    if rgb.dim() != 4 or rgb.shape[1] != 3 or not rgb.is_contiguous():
        raise ValueError("rgb must be a contiguous [N, 3, H, W] tensor")
    n, _, h, w = rgb.shape
    if out is None:
        out = empty_qmap(n, 1, h, w, rgb.dtype, rgb.device)
    elif not is_device_layout(out) or tuple(out.shape) != (n, 4, 1, h, w) or out.dtype != rgb.dtype:
        raise ValueError("out must be [N, 4, 1, H, W] in device layout with rgb's dtype")
    with torch.cuda.device(rgb.device):
        rc = lib.quan_poincare_map(_ptr(rgb), _ptr(out), n, h, w, _dtype_code(rgb), _stream(rgb.device))
    _check(rc)
    return out


def quan_qconv2d_poincare_forward(rgb, packed, weight_shape, bias=None, stride=1, pad=0, dilation=1, out=None):
    """The stem convolution on RGB images [N, 3, H, W] (contiguous) with the
    Poincare map (eq. 4) fused into its loads: equals quan_qconv2d_forward_packed
    of quan_poincare_map(rgb).  weight_shape: (Cout, 1, kh, kw) of the packed
    kernels.  Returns out [N, 4, Cout, Ho, Wo] in device layout."""
    lib = load_library()
    if rgb.dim() != 4 or rgb.shape[1] != 3 or not rgb.is_contiguous():
        raise ValueError("rgb must be a contiguous [N, 3, H, W] tensor")
    n, _, h, w = rgb.shape
    c_out, c_in, k_h, k_w = (int(v) for v in weight_shape)
    if c_in != 1:
        raise ValueError("the Poincare stem has one input quaternion channel (weight_shape[1] == 1)")
    if bias is not None and (tuple(bias.shape) != (4, c_out) or not bias.is_contiguous()
                             or bias.dtype != rgb.dtype or bias.device != rgb.device):
        raise ValueError("bias must be a contiguous [4, Cout] tensor like rgb")
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    dh, dw = _pair(dilation)
    ho, wo = conv_out_size(h, k_h, sh, ph, dh), conv_out_size(w, k_w, sw, pw, dw)
    if out is None:
        out = empty_qmap(n, c_out, ho, wo, rgb.dtype, rgb.device)
    elif not is_device_layout(out) or tuple(out.shape) != (n, 4, c_out, ho, wo) or out.dtype != rgb.dtype:
        raise ValueError("out must be [N, 4, Cout, Ho, Wo] in device layout with rgb's dtype")
    with torch.cuda.device(rgb.device):
        rc = lib.quan_qconv2d_poincare_forward(_ptr(rgb), _ptr(packed), _ptr(bias), sh, sw, ph, pw, dh, dw,
                                               _ptr(out), n, h, w, c_out, k_h, k_w, _dtype_code(rgb),
                                               _stream(rgb.device))
    _check(rc)
    return out


def quan_qconv2d_backward_data(dy, w_r, w_i, w_j, w_k, input_hw, stride=1, pad=0, dilation=1, dx=None,
                               _fn="quan_qconv2d_backward_data"):
    """Input gradient of quan_qconv2d_forward for dL/dY = dy ([N, 4, Cout, Ho,
    Wo], device layout); input_hw = (H, W) of the forward input.  Returns dx
    [N, 4, Cin, H, W] in device layout."""
    lib = load_library()
    if not is_device_layout(dy):
        raise ValueError("dy must be [N, 4, Cout, Ho, Wo] in device layout")
    c_out, c_in, k_h, k_w = _check_weights((w_r, w_i, w_j, w_k), dy)
    n, _, c_out_y, ho, wo = dy.shape
    if c_out_y != c_out:
        raise ValueError("dy's channels do not match the kernels")
    h, w = (int(v) for v in input_hw)
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    dh, dw = _pair(dilation)
    if (conv_out_size(h, k_h, sh, ph, dh), conv_out_size(w, k_w, sw, pw, dw)) != (ho, wo):
        raise ValueError("input_hw does not give dy's spatial size")
    if dx is None:
        dx = empty_qmap(n, c_in, h, w, dy.dtype, dy.device)
    elif not is_device_layout(dx) or tuple(dx.shape) != (n, 4, c_in, h, w) or dx.dtype != dy.dtype:
        raise ValueError("dx must be [N, 4, Cin, H, W] in device layout with dy's dtype")
    with torch.cuda.device(dy.device):
        rc = getattr(lib, _fn)(_ptr(dy), _ptr(w_r), _ptr(w_i), _ptr(w_j), _ptr(w_k), sh, sw, ph, pw,
                               dh, dw, _ptr(dx), n, c_in, h, w, c_out, k_h, k_w, _dtype_code(dy),
                               _stream(dy.device))
    _check(rc)
    return dx


def quan_qconv2d_backward_weight(x, dy, kernel_hw, stride=1, pad=0, dilation=1, with_bias=True,
                                 _fn="quan_qconv2d_backward_weight"):
    """Weight (and bias) gradients of quan_qconv2d_forward for dL/dY = dy:
    returns ([dW_r, dW_i, dW_j, dW_k] each fp32 [Cout, Cin, kh, kw], db fp32
    [4, Cout] or None)."""
    lib = load_library()
    for name, t in (("x", x), ("dy", dy)):
        if not is_device_layout(t):
            raise ValueError(f"{name} must be in device layout")
    if dy.dtype != x.dtype or dy.device != x.device:
        raise ValueError("x and dy must share dtype and device")
    n, _, c_in, h, w = x.shape
    c_out = dy.shape[2]
    k_h, k_w = (int(v) for v in kernel_hw)
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    dh, dw_ = _pair(dilation)
    if tuple(dy.shape) != (n, 4, c_out, conv_out_size(h, k_h, sh, ph, dh), conv_out_size(w, k_w, sw, pw, dw_)):
        raise ValueError("dy's shape does not match x and the layer geometry")
    dws = [torch.empty((c_out, c_in, k_h, k_w), dtype=torch.float32, device=x.device) for _ in range(4)]
    db = torch.empty((4, c_out), dtype=torch.float32, device=x.device) if with_bias else None
    with torch.cuda.device(x.device):
        rc = getattr(lib, _fn)(_ptr(x), _ptr(dy), sh, sw, ph, pw, dh, dw_, *[_ptr(t) for t in dws],
                               _ptr(db), n, c_in, h, w, c_out, k_h, k_w, _dtype_code(x),
                               _stream(x.device))
    _check(rc)
    return dws, db


def quan_qconv2d_separable_backward_data(dy, w_r, w_i, w_j, w_k, input_hw, stride=1, pad=0, dilation=1, dx=None):
    """Input gradient of quan_qconv2d_separable_forward (eqs. 8-10); arguments
    and result as in quan_qconv2d_backward_data."""
    return quan_qconv2d_backward_data(dy, w_r, w_i, w_j, w_k, input_hw, stride, pad, dilation, dx,
                                      _fn="quan_qconv2d_separable_backward_data")


def quan_qconv2d_separable_backward_weight(x, dy, kernel_hw, stride=1, pad=0, dilation=1, with_bias=True):
    """Weight (and bias) gradients of quan_qconv2d_separable_forward (eqs.
    8-10); arguments and result as in quan_qconv2d_backward_weight."""
    return quan_qconv2d_backward_weight(x, dy, kernel_hw, stride, pad, dilation, with_bias,
                                        _fn="quan_qconv2d_separable_backward_weight")


def quan_iqbn_backward(x, dout, mean, var, gamma, y=None, eps=1e-5, dx=None):
    """Gradient of training-mode IQBN (+ ReLU when the forward output y is
    given) for dL/dout = dout, with the forward's saved batch statistics.
    Returns (dx, dgamma, dbeta)."""
    lib = load_library()
    for name, t in (("x", x), ("dout", dout)) + ((("y", y),) if y is not None else ()):
        if not is_device_layout(t) or t.shape != x.shape or t.dtype != x.dtype:
            raise ValueError(f"{name} must be [N, 4, C, H, W] in device layout like x")
    n, _, c, h, w = x.shape
    for name, t in (("mean", mean), ("var", var), ("gamma", gamma)):
        if tuple(t.shape) != (4, c) or t.dtype != torch.float32 or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous float32 [4, C] tensor")
    if dx is None:
        dx = empty_qmap(n, c, h, w, x.dtype, x.device)
    elif not is_device_layout(dx) or dx.shape != x.shape or dx.dtype != x.dtype:
        raise ValueError("dx must be [N, 4, C, H, W] in device layout like x")
    dgamma = torch.empty(4, c, dtype=torch.float32, device=x.device)
    dbeta = torch.empty(4, c, dtype=torch.float32, device=x.device)
    with torch.cuda.device(x.device):
        rc = lib.quan_iqbn_backward(_ptr(x), _ptr(dout), _ptr(y), _ptr(mean), _ptr(var), _ptr(gamma),
                                    float(eps), _ptr(dx), _ptr(dgamma), _ptr(dbeta), n, c, h, w,
                                    _dtype_code(x), _stream(x.device))
    _check(rc)
    return dx, dgamma, dbeta


def _iqbn(fn_name, x, gamma, beta, eps, out, mean, var):
    lib = load_library()
    if not is_device_layout(x):
        raise ValueError("x must be [N, 4, C, H, W] stored channels-last by component")
    n, _, c, h, w = x.shape
    for name, t in (("gamma", gamma), ("beta", beta)):
        if tuple(t.shape) != (4, c) or t.dtype != torch.float32 or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous float32 [4, C] tensor")
    if out is None:
        out = empty_qmap(n, c, h, w, x.dtype, x.device)
    elif not is_device_layout(out) or out.shape != x.shape or out.dtype != x.dtype:
        raise ValueError("out must match x (device layout)")
    if mean is None:
        mean = torch.empty(4, c, dtype=torch.float32, device=x.device)
    if var is None:
        var = torch.empty(4, c, dtype=torch.float32, device=x.device)
    with torch.cuda.device(x.device):
        rc = getattr(lib, fn_name)(_ptr(x), _ptr(gamma), _ptr(beta), float(eps), _ptr(out),
                                   _ptr(mean), _ptr(var), n, c, h, w, _dtype_code(x),
                                   _stream(x.device))
    _check(rc)
    return out, mean, var


def _iqbn_desc(fn_name, x, gamma, beta, eps, out, mean, var):
    lib = load_library()
    if x.dim() != 5:
        raise ValueError("x must be [N, 4, C, H, W]")
    n, _, c, h, w = x.shape
    if out is None:
        out = empty_qmap(n, c, h, w, x.dtype, x.device)
    if mean is None:
        mean = torch.empty(4, c, dtype=torch.float32, device=x.device)
    if var is None:
        var = torch.empty(4, c, dtype=torch.float32, device=x.device)
    for t in (gamma, beta, out, mean, var):
        if t.device != x.device:
            raise ValueError("all tensors must be on x's device")
    descs = [describe(t) for t in (x, gamma, beta, out, mean, var)]
    with torch.cuda.device(x.device):
        rc = getattr(lib, fn_name)(_ref(descs[0]), _ref(descs[1]), _ref(descs[2]), float(eps),
                                   _ref(descs[3]), _ref(descs[4]), _ref(descs[5]), _stream(x.device))
    _check(rc)
    return out, mean, var


def quan_iqbn_forward(x, gamma, beta, eps=1e-5, out=None, mean=None, var=None):
    """IQBN (Section III-C, eqs. 11/12).  Returns (out, mean, var).  Tensors
    go to the library as descriptors; it checks their shapes and layouts."""
    return _iqbn_desc("quan_iqbn_forward_desc", x, gamma, beta, eps, out, mean, var)


def quan_iqbn_relu_forward(x, gamma, beta, eps=1e-5, out=None, mean=None, var=None):
    """IQBN followed by a component-wise ReLU.  Returns (out, mean, var)."""
    return _iqbn_desc("quan_iqbn_relu_forward_desc", x, gamma, beta, eps, out, mean, var)


def quan_iqbn_forward_noalloc(x, gamma, beta, eps=1e-5, out=None, mean=None, var=None):
    """IQBN with the partial statistics in the library's fixed per-GPU scratch
    array (no device allocation by the call; out, mean and var must then be
    passed in for an allocation-free call).  Returns (out, mean, var)."""
    return _iqbn("quan_iqbn_forward_noalloc", x, gamma, beta, eps, out, mean, var)


def quan_last_error() -> str:
    return load_library().quan_last_error().decode()


def quan_release() -> None:
    _check(load_library().quan_release())


def quan_version() -> str:
    return load_library().quan_version().decode()
