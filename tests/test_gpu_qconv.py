"""GPU parity of quan_qconv2d_forward against the CPU oracle, through the C ABI.

Shapes span several work-group tiles with ragged tails in every dimension
(pixels, output channels, input channels), strides, pads, dilations and
kernel sizes; both dtypes.  Outputs are pre-filled with NaN so an unwritten
element fails the comparison."""
import numpy as np
import pytest
import torch

import oracle
from paper_2509_05512_amd import quan
from parity import assert_close, f64, say

pytestmark = pytest.mark.gpu

DT = {"fp32": torch.float32, "bf16": torch.bfloat16}

# (N, Cin, Cout, H, W, k, stride, pad, dilation)
SHAPES = [
    (2, 4, 4, 16, 16, 3, 1, 1, 1),      # the tiny fp32 layer's geometry
    (3, 8, 16, 9, 11, 3, 1, 1, 1),
    (2, 16, 64, 13, 10, 3, 2, 1, 1),    # stride 2
    (1, 32, 80, 12, 12, 3, 1, 2, 2),    # dilation 2, ragged output-channel tile
    (2, 5, 7, 9, 9, 3, 1, 1, 1),        # channels not a multiple of the vector width
    (1, 3, 3, 7, 5, 5, 1, 2, 1),        # 5x5, tiny
    (2, 64, 64, 15, 15, 1, 1, 0, 1),    # 1x1
    (1, 24, 40, 17, 19, 3, 2, 0, 1),    # pad 0, stride 2, ragged input-channel block
    (4, 16, 16, 20, 18, 3, 1, 1, 1),
    (1, 48, 128, 11, 7, 3, 1, 1, 1),    # several output-channel tiles
    (3, 2, 1, 6, 6, 3, 1, 1, 1),        # single output channel
    (1, 1, 2, 5, 4, 1, 2, 0, 1),        # single input channel, 1x1 stride 2
    (2, 128, 64, 9, 10, 3, 1, 1, 1),    # one component per K stage, two channel blocks
    (1, 96, 48, 11, 9, 3, 2, 1, 1),     # two components per K stage, three channel blocks
    (1, 64, 256, 7, 8, 3, 1, 1, 1),     # one component per stage, four output-channel tiles
    (3, 40, 24, 6, 7, 3, 1, 1, 2),      # ragged channel block, dilation 2
]


def _case(shape, dtype, seed, with_bias=True):
    N, Cin, Cout, H, W, k, s, p, d = shape
    rng = np.random.default_rng(seed)
    x = torch.from_numpy(rng.standard_normal((N, 4, Cin, H, W), dtype=np.float32)).to(dtype)
    w = torch.from_numpy((rng.standard_normal((4, Cout, Cin, k, k), dtype=np.float32)
                          / np.float32(np.sqrt(4 * Cin * k * k)))).to(dtype)
    b = torch.from_numpy(rng.standard_normal((4, Cout), dtype=np.float32) * np.float32(0.1)).to(dtype) \
        if with_bias else None
    return x, w, b


def _run_gpu(x, w, b, s, p, d, poison=True):
    dev = torch.device("cuda:0")
    xg = quan.to_device_layout(x.to(dev))
    wg = [w[q].contiguous().to(dev) for q in range(4)]
    bg = b.contiguous().to(dev) if b is not None else None
    N, _, Cin, H, W = x.shape
    Cout, k = w.shape[1], w.shape[3]
    ho, wo = quan.conv_out_size(H, k, s, p, d), quan.conv_out_size(W, k, s, p, d)
    out = quan.empty_qmap(N, Cout, ho, wo, x.dtype, dev)
    if poison:
        out.fill_(float("nan"))
    quan.quan_qconv2d_forward(xg, *wg, bias=bg, stride=s, pad=p, dilation=d, out=out)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_qconv2d_matches_oracle(shape, dtype):
    say(f"qconv2d parity {dtype} {shape}")
    dt = DT[dtype]
    x, w, b = _case(shape, dt, seed=hash(shape) % 1000)
    N, Cin, Cout, H, W, k, s, p, d = shape
    out = _run_gpu(x, w, b, s, p, d)
    ref = oracle.qconv2d(f64(x), f64(w), f64(b), s, p, d)
    assert_close(f64(out), ref, dt, f"qconv2d {dtype} {shape}")


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_qconv2d_without_bias(dtype):
    shape = (2, 16, 32, 10, 9, 3, 1, 1, 1)
    say(f"qconv2d no-bias {dtype}")
    dt = DT[dtype]
    x, w, _ = _case(shape, dt, seed=5, with_bias=False)
    out = _run_gpu(x, w, None, 1, 1, 1)
    ref = oracle.qconv2d(f64(x), f64(w), None, 1, 1, 1)
    assert_close(f64(out), ref, dt, "no bias")


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_identity_kernel_returns_input_exactly(dtype):
    say(f"qconv2d identity {dtype}")
    dt = DT[dtype]
    N, C, H, W = 2, 16, 9, 7
    x = torch.randn(N, 4, C, H, W, generator=torch.Generator().manual_seed(3)).to(dt)
    w = torch.zeros(4, C, C, 3, 3, dtype=dt)
    for c in range(C):
        w[0, c, c, 1, 1] = 1
    out = _run_gpu(x, w, None, 1, 1, 1)
    assert torch.equal(out.cpu(), x), "identity kernel must reproduce the input bit for bit"


def test_orientation_i_times_j_is_k():
    say("qconv2d orientation")
    x = torch.zeros(1, 4, 1, 1, 1, dtype=torch.float32)
    x[0, 2] = 1.0                      # X = j
    w = torch.zeros(4, 1, 1, 1, 1)
    w[1] = 1.0                         # W = i
    out = _run_gpu(x, w, None, 1, 0, 1).cpu().reshape(4)
    assert torch.equal(out, torch.tensor([0.0, 0.0, 0.0, 1.0]))


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_deterministic(dtype):
    say(f"qconv2d determinism {dtype}")
    dt = DT[dtype]
    x, w, b = _case((2, 32, 64, 14, 14, 3, 1, 1, 1), dt, seed=9)
    o1 = _run_gpu(x, w, b, 1, 1, 1).cpu()
    o2 = _run_gpu(x, w, b, 1, 1, 1).cpu()
    assert torch.equal(o1, o2)


def test_library_rejects_wrong_layout():
    # the descriptors carry torch's real strides; the library refuses them
    say("qconv2d / iqbn layout rejection")
    dev = torch.device("cuda:0")
    x = torch.randn(1, 4, 4, 5, 5, device=dev)          # plain contiguous: wrong layout
    w = [torch.randn(4, 4, 3, 3, device=dev) for _ in range(4)]
    with pytest.raises(quan.QuanError) as ei:
        quan.quan_qconv2d_forward(x, *w, stride=1, pad=1)
    assert ei.value.code == quan.QUAN_ERR_LAYOUT
    g = torch.ones(4, 4, device=dev)
    with pytest.raises(quan.QuanError) as ei:
        quan.quan_iqbn_forward(x, g, g)
    assert ei.value.code == quan.QUAN_ERR_LAYOUT
    wt = [t.permute(0, 2, 3, 1).contiguous().permute(0, 3, 1, 2) for t in w]   # OHWI memory
    with pytest.raises(quan.QuanError) as ei:
        quan.quan_qconv2d_forward(quan.to_device_layout(x), *wt, stride=1, pad=1)
    assert ei.value.code == quan.QUAN_ERR_LAYOUT


def test_abi_error_from_device_tensors():
    say("qconv2d ABI error path")
    dev = torch.device("cuda:0")
    x = quan.to_device_layout(torch.randn(1, 4, 4, 3, 3, device=dev))
    w = [torch.randn(4, 4, 5, 5, device=dev) for _ in range(4)]
    with pytest.raises(quan.QuanError) as ei:
        quan.quan_qconv2d_forward(x, *w, stride=1, pad=0)   # 5x5 kernel on a 3x3 image
    assert ei.value.code == -2


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_packed_path_equals_forward(dtype):
    """Weights packed once, then quan_qconv2d_forward_packed twice (two
    shapes), bit-identical to quan_qconv2d_forward."""
    say(f"qconv2d packed path {dtype}")
    dt = DT[dtype]
    dev = torch.device("cuda:0")
    x, w, b = _case((2, 24, 72, 11, 13, 3, 1, 1, 1), dt, seed=21)
    wg = [w[q].contiguous().to(dev) for q in range(4)]
    bg = b.to(dev)
    packed = quan.quan_qconv2d_pack_weights(*wg)
    assert packed.numel() == quan.quan_qconv2d_packed_bytes(24, 72, 3, 3, dt)
    for xs, s in ((x, 1), (x[:1, :, :, :7, :9].contiguous(), 2)):
        xg = quan.to_device_layout(xs.to(dev))
        ref = quan.quan_qconv2d_forward(xg, *wg, bias=bg, stride=s, pad=1)
        got = quan.quan_qconv2d_forward_packed(xg, packed, tuple(wg[0].shape), bias=bg, stride=s, pad=1)
        torch.cuda.synchronize()
        assert torch.equal(got.cpu(), ref.cpu())


def test_descriptor_unit_axis_takes_any_stride():
    """An axis of extent 1 is never stepped: the library accepts any stride
    for it, and the result is the one of the dense tensor."""
    say("descriptor: extent-1 axis with an odd stride")
    dev = torch.device("cuda:0")
    g = torch.Generator().manual_seed(5)
    x = quan.to_device_layout(torch.randn(1, 4, 8, 9, 7, generator=g).to(torch.bfloat16).to(dev))
    w = [(torch.randn(8, 8, 3, 3, generator=g) * 0.1).to(torch.bfloat16).to(dev) for _ in range(4)]
    x_odd = x.as_strided(x.shape, (12345,) + tuple(x.stride()[1:]))
    y_ref = quan.quan_qconv2d_forward(x, *w, stride=1, pad=1)
    y_odd = quan.quan_qconv2d_forward(x_odd, *w, stride=1, pad=1)
    torch.cuda.synchronize()
    assert torch.equal(y_ref.cpu(), y_odd.cpu())
    gm, bt = torch.ones(4, 8, device=dev), torch.zeros(4, 8, device=dev)
    o_ref, m_ref, v_ref = quan.quan_iqbn_forward(x, gm, bt)
    o_odd, m_odd, v_odd = quan.quan_iqbn_forward(x_odd, gm, bt)
    torch.cuda.synchronize()
    assert torch.equal(o_ref.cpu(), o_odd.cpu()) and torch.equal(m_ref.cpu(), m_odd.cpu())
