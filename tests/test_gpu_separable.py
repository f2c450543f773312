"""GPU parity of the separable QUAN convolution (Section III-B, eq. 7)
against the oracle's fp64 separable convolution, through the C ABI: shapes
spanning several tiles with ragged tails, strides, pads, dilations, channel
counts off the vector width, both dtypes; the packed entry point; the full
imagenet_stage layer on sampled pixels; and the properties eq. 7 fixes (row
r equals the Hamilton product's, the identity kernel copies x_r to every
component).  Outputs are pre-filled with NaN so an unwritten element fails."""
import numpy as np
import pytest
import torch

import oracle
from paper_2509_05512_amd import quan
from parity import assert_close, conv_reference_sampled, f64, sample_pixels, say

pytestmark = pytest.mark.gpu

DT = {"fp32": torch.float32, "bf16": torch.bfloat16}

# (N, Cin, Cout, H, W, k, stride, pad, dilation)
SHAPES = [
    (2, 4, 4, 16, 16, 3, 1, 1, 1),
    (3, 8, 16, 9, 11, 3, 1, 1, 1),
    (2, 16, 64, 13, 10, 3, 2, 1, 1),    # stride 2
    (1, 32, 80, 12, 12, 3, 1, 2, 2),    # dilation 2, ragged output-channel tile
    (2, 5, 7, 9, 9, 3, 1, 1, 1),        # channels not a multiple of the vector width
    (2, 64, 64, 15, 15, 1, 1, 0, 1),    # 1x1
    (1, 24, 40, 17, 19, 3, 2, 0, 1),    # ragged input-channel block
    (3, 2, 1, 6, 6, 3, 1, 1, 1),        # single output channel
    (2, 128, 64, 9, 10, 3, 1, 1, 1),    # several channel blocks per tap
    (1, 64, 256, 7, 8, 3, 1, 1, 1),     # several output-channel tiles
]


def _case(shape, dtype, seed):
    N, Cin, Cout, H, W, k, s, p, d = shape
    rng = np.random.default_rng(seed)
    x = torch.from_numpy(rng.standard_normal((N, 4, Cin, H, W), dtype=np.float32)).to(dtype)
    w = torch.from_numpy((rng.standard_normal((4, Cout, Cin, k, k), dtype=np.float32)
                          / np.float32(np.sqrt(Cin * k * k)))).to(dtype)
    b = torch.from_numpy(rng.standard_normal((4, Cout), dtype=np.float32) * np.float32(0.1)).to(dtype)
    return x, w, b


def _out(x, w, s, p, d):
    N, _, Cin, H, W = x.shape
    Cout, k = w.shape[1], w.shape[3]
    ho, wo = quan.conv_out_size(H, k, s, p, d), quan.conv_out_size(W, k, s, p, d)
    out = quan.empty_qmap(N, Cout, ho, wo, x.dtype, torch.device("cuda:0"))
    out.fill_(float("nan"))
    return out


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_separable_matches_oracle(shape, dtype):
    say(f"separable parity {dtype} {shape}")
    dt = DT[dtype]
    x, w, b = _case(shape, dt, seed=hash(shape) % 1000)
    N, Cin, Cout, H, W, k, s, p, d = shape
    dev = torch.device("cuda:0")
    out = _out(x, w, s, p, d)
    quan.quan_qconv2d_separable_forward(quan.to_device_layout(x.to(dev)), *[w[q].contiguous().to(dev) for q in range(4)],
                                        bias=b.to(dev), stride=s, pad=p, dilation=d, out=out)
    torch.cuda.synchronize()
    ref = oracle.qconv2d_separable(f64(x), f64(w), f64(b), s, p, d)
    assert_close(f64(out), ref, dt, f"separable {dtype} {shape}")


def test_separable_packed_equals_unpacked():
    say("separable packed")
    shape = (2, 32, 64, 11, 13, 3, 1, 1, 1)
    x, w, b = _case(shape, torch.bfloat16, seed=3)
    dev = torch.device("cuda:0")
    xg = quan.to_device_layout(x.to(dev))
    wg = [w[q].contiguous().to(dev) for q in range(4)]
    packed = quan.quan_qconv2d_pack_weights(*wg)
    y1 = quan.quan_qconv2d_separable_forward(xg, *wg, bias=b.to(dev), stride=1, pad=1)
    y2 = quan.quan_qconv2d_separable_forward_packed(xg, packed, tuple(wg[0].shape), bias=b.to(dev), stride=1,
                                                    pad=1)
    torch.cuda.synchronize()
    assert torch.equal(y1.cpu(), y2.cpu())


def test_separable_real_row_equals_hamilton():
    """Row r of eq. 7 is row r of the Hamilton product: the two GPU kernels
    agree on the real component (fp32, to rounding)."""
    say("separable row r vs hamilton")
    shape = (2, 16, 32, 9, 10, 3, 1, 1, 1)
    x, w, b = _case(shape, torch.float32, seed=4)
    dev = torch.device("cuda:0")
    xg = quan.to_device_layout(x.to(dev))
    wg = [w[q].contiguous().to(dev) for q in range(4)]
    ys = quan.quan_qconv2d_separable_forward(xg, *wg, bias=b.to(dev), stride=1, pad=1)
    yh = quan.quan_qconv2d_forward(xg, *wg, bias=b.to(dev), stride=1, pad=1)
    torch.cuda.synchronize()
    assert_close(f64(ys.cpu())[:, 0], f64(yh.cpu())[:, 0], torch.float32, "row r")


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_separable_identity_kernel_copies_real_part(dtype):
    """W_r = identity, W_i = W_j = W_k = 0: every output component is x_r
    (eq. 7 has +W_r x_r in every row), exactly."""
    say(f"separable identity {dtype}")
    dt = DT[dtype]
    N, C, H, W = 2, 24, 9, 7
    rng = np.random.default_rng(9)
    x = torch.from_numpy(rng.standard_normal((N, 4, C, H, W), dtype=np.float32)).to(dt)
    w = torch.zeros((4, C, C, 3, 3), dtype=dt)
    for c in range(C):
        w[0, c, c, 1, 1] = 1.0
    dev = torch.device("cuda:0")
    y = quan.quan_qconv2d_separable_forward(quan.to_device_layout(x.to(dev)), *[w[q].contiguous().to(dev) for q in range(4)],
                                            stride=1, pad=1)
    torch.cuda.synchronize()
    yc = y.cpu()
    for p in range(4):
        assert torch.equal(yc[:, p], x[:, 0]), p


def test_separable_full_imagenet_layer_sampled():
    """The imagenet_stage layer (64x56x56, 64->64) on the persistent grid:
    sampled output pixels (all channels and components) against the oracle."""
    say("separable full-size sampled")
    from paper_2509_05512_amd import workloads
    wl = workloads.WORKLOADS["imagenet_stage"]
    tens = workloads.generate(wl)
    layer = tens.layers[0]
    dev = torch.device("cuda:0")
    xg = quan.to_device_layout(tens.x.to(dev))
    wg = [layer.weight[q].contiguous().to(dev) for q in range(4)]
    y = quan.quan_qconv2d_separable_forward(xg, *wg, stride=1, pad=1)
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    n, ho, wo = wl.n, wl.h, wl.w
    samples = sample_pixels(rng, n, ho, wo, 48)
    ref = conv_reference_sampled(f64(tens.x), f64(layer.weight), None, 1, 1, 1, 3, samples,
                                 conv=oracle.qconv2d_separable)
    yc = y.cpu()
    got = np.stack([f64(yc[nn, :, :, oy, ox]) for (nn, oy, ox) in samples])
    assert_close(got, ref, torch.bfloat16, "separable imagenet_stage sampled")
