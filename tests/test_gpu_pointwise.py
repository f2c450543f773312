"""GPU parity of the pointwise (1x1) streaming convolution kernel, which runs
every bf16 1x1 Hamilton layer without padding with 32 or 64 input and
output channels: the signed weights stay in registers, activations stream
through LDS in 32-pixel stages, and each work-group takes an equal run of
consecutive stages (ceil(stages / 256) on 256 compute units).

Every case is compared in full against the oracle: all four channel
combinations, a ragged last stage, a single stage of fewer than 32 pixels,
stride 2 (a gathered input), runs long enough to wrap the stage ring (8
slots at 64 input channels, 16 at 32), the full 16 x 80 x 80 layer of the
detection-shaped pair; the IQBN statistics gathered per work-group in the
epilogue (and the separate pass), the folded inference epilogue, the input
gradient of a 1x1 layer (itself a 1x1 convolution), and launches on two
streams."""
import numpy as np
import pytest
import torch

import oracle
from paper_2509_05512_amd import quan
from parity import assert_close, f64, say

pytestmark = pytest.mark.gpu

BF16 = torch.bfloat16


def stages_per_group(pixels, cus=256):
    stages = -(-pixels // 32)
    return -(-stages // cus)


# (N, Cin, Cout, H, W, stride)
CONV_CASES = [
    (8, 64, 64, 64, 80, 1),     # 40960 px: 5 stages per work-group, all full
    (3, 64, 64, 37, 41, 1),     # 4551 px: one stage each, the last one 7 px
    (1, 64, 64, 3, 5, 1),       # 15 px: one work-group, one partial stage
    (8, 32, 64, 50, 50, 1),     # 20000 px: 3 stages per work-group, the last group 1
    (8, 64, 32, 50, 50, 1),
    (8, 32, 32, 50, 50, 1),
    (4, 64, 64, 81, 79, 2),     # stride 2: 41 x 40 outputs gathered from 81 x 79
    (16, 64, 64, 80, 80, 1),    # 102400 px: 13 stages per group (the ring of 8 wraps), last group 2
    (16, 32, 64, 96, 96, 1),    # 147456 px: 18 stages per group (the ring of 16 wraps)
    (5, 32, 32, 71, 53, 3),     # stride 3, ragged
]


def _inputs(case, seed):
    N, Cin, Cout, H, W = case[:5]
    rng = np.random.default_rng(seed)
    x = torch.from_numpy(rng.standard_normal((N, 4, Cin, H, W), dtype=np.float32)).to(BF16)
    w = torch.from_numpy(rng.standard_normal((4, Cout, Cin, 1, 1), dtype=np.float32)
                         / np.float32(np.sqrt(4 * Cin))).to(BF16)
    b = torch.from_numpy(rng.standard_normal((4, Cout), dtype=np.float32) * np.float32(0.3)).to(BF16)
    return x, w, b


def _label(case):
    N, Cin, Cout, H, W, s = case
    ho, wo = quan.conv_out_size(H, 1, s, 0, 1), quan.conv_out_size(W, 1, s, 0, 1)
    px = N * ho * wo
    return f"{case} pixels={px} stages_per_group={stages_per_group(px)}"


def _conv(x, w, b, s, stream=None):
    dev = torch.device("cuda:0")
    N, _, Cin, H, W = x.shape
    Cout = w.shape[1]
    ho, wo = quan.conv_out_size(H, 1, s, 0, 1), quan.conv_out_size(W, 1, s, 0, 1)
    out = quan.empty_qmap(N, Cout, ho, wo, BF16, dev)
    out.fill_(float("nan"))
    quan.quan_qconv2d_forward(quan.to_device_layout(x.to(dev)), *[w[q].contiguous().to(dev) for q in range(4)],
                              bias=b.to(dev), stride=s, pad=0, out=out)
    return out


@pytest.mark.parametrize("case", CONV_CASES, ids=[str(c) for c in CONV_CASES])
def test_pointwise_conv_matches_oracle(case):
    label = _label(case)
    say(f"pointwise conv {label}")
    x, w, b = _inputs(case, seed=sum(case))
    out = _conv(x, w, b, case[5])
    torch.cuda.synchronize()
    assert_close(f64(out), oracle.qconv2d(f64(x), f64(w), f64(b), case[5], 0, 1), BF16, f"pointwise {label}")


def test_pointwise_conv_without_bias():
    case = (3, 64, 64, 37, 41, 1)
    say(f"pointwise conv without bias {_label(case)}")
    x, w, _ = _inputs(case, seed=3)
    dev = torch.device("cuda:0")
    out = quan.quan_qconv2d_forward(quan.to_device_layout(x.to(dev)), *[w[q].contiguous().to(dev) for q in range(4)])
    torch.cuda.synchronize()
    assert_close(f64(out), oracle.qconv2d(f64(x), f64(w), None, 1, 0, 1), BF16, "pointwise no bias")


STAT_CASES = [(3, 64, 64, 37, 41, 1), (16, 64, 64, 80, 80, 1), (8, 32, 32, 50, 50, 1)]


@pytest.mark.parametrize("relu", [False, True])
@pytest.mark.parametrize("stats", ["epilogue", "pass"])
@pytest.mark.parametrize("case", STAT_CASES, ids=[str(c) for c in STAT_CASES])
def test_pointwise_statistics(case, stats, relu):
    """Convolution + IQBN: the conv output against the oracle convolution,
    and out / mean / var against the oracle's IQBN of that GPU conv output
    (the epilogue's per-work-group runs include a short last run)."""
    label = f"{_label(case)} stats={stats} relu={relu}"
    say(f"pointwise statistics {label}")
    N, Cin, Cout, H, W, s = case
    x, w, b = _inputs(case, seed=177 + relu)
    rng = np.random.default_rng(178)
    g = torch.from_numpy(rng.uniform(0.5, 1.5, (4, Cout)).astype(np.float32))
    be = torch.from_numpy((rng.standard_normal((4, Cout)) * 0.2).astype(np.float32))
    dev = torch.device("cuda:0")
    xg = quan.to_device_layout(x.to(dev))
    wg = [w[q].contiguous().to(dev) for q in range(4)]
    packed = quan.quan_qconv2d_pack_weights(*wg)
    shape = tuple(wg[0].shape)
    conv = quan.quan_qconv2d_forward_packed(xg, packed, shape, bias=b.to(dev), stride=s)
    out, mean, var = quan.quan_qconv2d_iqbn_forward(xg, packed, shape, g.to(dev), be.to(dev), bias=b.to(dev),
                                                     stride=s, relu=relu, stats=stats)
    torch.cuda.synchronize()
    conv, out, mean, var = conv.cpu(), out.cpu(), mean.cpu(), var.cpu()
    assert_close(f64(conv), oracle.qconv2d(f64(x), f64(w), f64(b), s, 0, 1), BF16, f"pointwise conv {label}")
    ref_out, ref_mean, ref_var = oracle.iqbn(f64(conv), f64(g), f64(be), 1e-5, relu)
    assert_close(mean.double().numpy(), ref_mean, torch.float32, f"mean {label}")
    assert_close(var.double().numpy(), ref_var, torch.float32, f"var {label}")
    assert_close(f64(out), ref_out, BF16, f"out {label}")


def test_pointwise_statistics_offset_columns():
    """Columns whose mean is large against their spread (bias 40, unit
    spread): the per-stage two-pass sums and the pairwise merge keep the
    variance where one-pass sums of squares would cancel."""
    case = (16, 64, 64, 80, 80, 1)
    say(f"pointwise statistics, offset columns {_label(case)}")
    N, Cin, Cout, H, W, s = case
    x, w, _ = _inputs(case, seed=12)
    b = torch.full((4, Cout), 40.0).to(BF16)
    g = torch.ones(4, Cout)
    be = torch.zeros(4, Cout)
    dev = torch.device("cuda:0")
    xg = quan.to_device_layout(x.to(dev))
    wg = [w[q].contiguous().to(dev) for q in range(4)]
    packed = quan.quan_qconv2d_pack_weights(*wg)
    shape = tuple(wg[0].shape)
    conv = quan.quan_qconv2d_forward_packed(xg, packed, shape, bias=b.to(dev))
    out, mean, var = quan.quan_qconv2d_iqbn_forward(xg, packed, shape, g.to(dev), be.to(dev), bias=b.to(dev),
                                                     stats="epilogue")
    torch.cuda.synchronize()
    ref_out, ref_mean, ref_var = oracle.iqbn(f64(conv.cpu()), f64(g), f64(be), 1e-5, False)
    assert_close(mean.cpu().double().numpy(), ref_mean, torch.float32, "offset mean")
    assert_close(var.cpu().double().numpy(), ref_var, torch.float32, "offset var")
    assert_close(f64(out.cpu()), ref_out, BF16, "offset out")


@pytest.mark.parametrize("relu", [False, True])
@pytest.mark.parametrize("case", [(3, 64, 64, 37, 41, 1), (16, 64, 64, 80, 80, 1), (8, 32, 64, 50, 50, 1)],
                         ids=str)
def test_pointwise_inference(case, relu):
    """The folded inference epilogue (stored statistics, eq. 12)."""
    label = f"{_label(case)} relu={relu}"
    say(f"pointwise inference {label}")
    N, Cin, Cout, H, W, s = case
    x, w, b = _inputs(case, seed=291 + relu)
    rng = np.random.default_rng(292)
    g = torch.from_numpy(rng.uniform(0.5, 1.5, (4, Cout)).astype(np.float32))
    be = torch.from_numpy((rng.standard_normal((4, Cout)) * 0.2).astype(np.float32))
    rm = torch.from_numpy((rng.standard_normal((4, Cout)) * 0.5).astype(np.float32))
    rv = torch.from_numpy(rng.uniform(0.5, 2.0, (4, Cout)).astype(np.float32))
    dev = torch.device("cuda:0")
    wg = [w[q].contiguous().to(dev) for q in range(4)]
    packed = quan.quan_qconv2d_pack_weights(*wg)
    out = quan.quan_qconv2d_iqbn_inference(quan.to_device_layout(x.to(dev)), packed, tuple(wg[0].shape),
                                           rm.to(dev), rv.to(dev), g.to(dev), be.to(dev), bias=b.to(dev),
                                           stride=s, relu=relu)
    torch.cuda.synchronize()
    ref = oracle.iqbn_inference(oracle.qconv2d(f64(x), f64(w), f64(b), s, 0, 1), f64(rm), f64(rv), f64(g),
                                f64(be), 1e-5, relu)
    assert_close(f64(out.cpu()), ref, BF16, f"pointwise inference {label}")


@pytest.mark.parametrize("case", [(4, 64, 64, 33, 35, 1), (4, 32, 64, 33, 35, 1)], ids=str)
def test_pointwise_backward_data(case):
    """The input gradient of a 1x1 layer is a 1x1 convolution of dy with the
    conjugate-transposed kernels: it runs on the pointwise kernel too."""
    label = _label(case)
    say(f"pointwise backward data {label}")
    N, Cin, Cout, H, W, s = case
    x, w, _ = _inputs(case, seed=401)
    rng = np.random.default_rng(402)
    dy = torch.from_numpy(rng.standard_normal((N, 4, Cout, H, W), dtype=np.float32)).to(BF16)
    dev = torch.device("cuda:0")
    dx = quan.quan_qconv2d_backward_data(quan.to_device_layout(dy.to(dev)),
                                         *[w[q].contiguous().to(dev) for q in range(4)], (H, W), stride=s)
    torch.cuda.synchronize()
    ref, _, _ = oracle.qconv2d_backward(f64(x), f64(w), f64(dy), s, 0, 1)
    assert_close(f64(dx.cpu()), ref, BF16, f"pointwise dX {label}")


def test_pointwise_two_streams():
    """Two layers launched on two streams at once, each into a NaN-filled
    output, both equal to the oracle."""
    say("pointwise two streams")
    cases = [(16, 64, 64, 80, 80, 1), (8, 32, 64, 50, 50, 1)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    data, outs = [], []
    for i, case in enumerate(cases):
        data.append(_inputs(case, seed=600 + i))
    torch.cuda.synchronize()
    for (x, w, b), case, st in zip(data, cases, streams):
        with torch.cuda.stream(st):
            outs.append(_conv(x, w, b, case[5]))
    torch.cuda.synchronize()
    for (x, w, b), case, out in zip(data, cases, outs):
        assert_close(f64(out.cpu()), oracle.qconv2d(f64(x), f64(w), f64(b), case[5], 0, 1), BF16,
                     f"two streams {_label(case)}")
