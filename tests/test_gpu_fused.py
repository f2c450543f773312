"""GPU parity of quan_qconv2d_iqbn_forward (convolution + IQBN) through the C
ABI, with the statistics gathered in the convolution's epilogue and in a
separate pass.

The fused call must equal its two-call composition: the convolution's output
is the same kernel's, so the oracle's IQBN applied to the GPU convolution
output (upcast to fp64) is the reference for out, mean and var, and the
convolution itself is checked against the oracle convolution on the same
inputs.  Shapes cover tiles with the fused statistics (>= 32 output channels,
whole 16-byte output chunks, ragged last pixel tile) and the layouts that
fall back to the separate IQBN passes."""
import numpy as np
import pytest
import torch

import oracle
from paper_2509_05512_amd import quan
from parity import assert_close, f64, say

pytestmark = pytest.mark.gpu

DT = {"fp32": torch.float32, "bf16": torch.bfloat16}

# (N, Cin, Cout, H, W, k, stride, pad, relu, dtype)
CASES = [
    (2, 16, 64, 13, 10, 3, 1, 1, False, "bf16"),   # 130 pixels per image: ragged last tile
    (3, 32, 64, 9, 11, 3, 2, 1, True, "bf16"),     # stride 2, ReLU
    (1, 64, 128, 12, 12, 1, 1, 0, False, "bf16"),  # 1x1, two output-channel tiles
    (4, 24, 32, 10, 10, 3, 1, 1, True, "bf16"),    # 32-channel tiles
    (2, 16, 72, 7, 9, 3, 1, 1, False, "bf16"),     # 72 = 64 + 8: partial channel tile
    (2, 32, 64, 10, 10, 1, 1, 0, True, "bf16"),    # two stages per tile
    (2, 16, 64, 8, 8, 1, 1, 0, False, "bf16"),     # one stage per tile
    (2, 8, 16, 9, 9, 3, 1, 1, True, "bf16"),       # 16 channels: separate IQBN passes
    (2, 8, 36, 6, 6, 3, 1, 1, False, "bf16"),      # c_out % 8 != 0: separate passes
    (2, 4, 4, 16, 16, 3, 1, 1, False, "fp32"),     # fp32: separate passes
]


def _case(case, seed):
    N, Cin, Cout, H, W, k, s, p, relu, dtype = case
    dt = DT[dtype]
    rng = np.random.default_rng(seed)
    x = torch.from_numpy(rng.standard_normal((N, 4, Cin, H, W), dtype=np.float32)).to(dt)
    w = torch.from_numpy(rng.standard_normal((4, Cout, Cin, k, k), dtype=np.float32)
                         / np.float32(np.sqrt(4 * Cin * k * k))).to(dt)
    b = torch.from_numpy(rng.standard_normal((4, Cout), dtype=np.float32) * np.float32(0.5)).to(dt)
    g = torch.from_numpy(rng.uniform(0.5, 1.5, (4, Cout)).astype(np.float32))
    be = torch.from_numpy((rng.standard_normal((4, Cout)) * 0.2).astype(np.float32))
    return x, w, b, g, be


def _gpu(x, w, b, g, be, s, p, relu, stats="epilogue"):
    dev = torch.device("cuda:0")
    xg = quan.to_device_layout(x.to(dev))
    wg = [w[q].contiguous().to(dev) for q in range(4)]
    packed = quan.quan_qconv2d_pack_weights(*wg)
    shape = tuple(wg[0].shape)
    bg, gg, beg = b.to(dev), g.to(dev), be.to(dev)
    conv = quan.quan_qconv2d_forward_packed(xg, packed, shape, bias=bg, stride=s, pad=p)
    out, mean, var = quan.quan_qconv2d_iqbn_forward(xg, packed, shape, gg, beg, bias=bg, stride=s,
                                                     pad=p, relu=relu, stats=stats)
    torch.cuda.synchronize()
    return conv.cpu(), out.cpu(), mean.cpu(), var.cpu()


@pytest.mark.parametrize("stats", ["epilogue", "pass"])
@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_fused_conv_iqbn_matches_oracle(case, stats):
    say(f"fused conv+iqbn {case} stats={stats}")
    N, Cin, Cout, H, W, k, s, p, relu, dtype = case
    dt = DT[dtype]
    x, w, b, g, be = _case(case, seed=sum(map(ord, str(case))) % 997)
    conv, out, mean, var = _gpu(x, w, b, g, be, s, p, relu, stats)
    # the convolution stage against the oracle convolution
    assert_close(f64(conv), oracle.qconv2d(f64(x), f64(w), f64(b), s, p, 1), dt, f"conv {case}")
    # the IQBN stage against the oracle IQBN of the GPU convolution output
    ref_out, ref_mean, ref_var = oracle.iqbn(f64(conv), f64(g), f64(be), 1e-5, relu)
    assert_close(mean.double().numpy(), ref_mean, torch.float32, f"mean {case}")
    assert_close(var.double().numpy(), ref_var, torch.float32, f"var {case}")
    assert_close(f64(out), ref_out, dt, f"out {case}")


@pytest.mark.parametrize("stats", ["epilogue", "pass", "auto"])
def test_fused_equals_separate_calls(stats):
    """The output of the convolution followed by quan_iqbn_forward, up to the
    statistics' summation order (last-ulp differences in mean/var)."""
    say(f"fused vs separate, stats={stats}")
    case = (2, 32, 64, 14, 14, 3, 1, 1, False, "bf16")
    x, w, b, g, be = _case(case, seed=7)
    dev = torch.device("cuda:0")
    conv, out, mean, var = _gpu(x, w, b, g, be, 1, 1, False, stats)
    out2, mean2, var2 = quan.quan_iqbn_forward(quan.to_device_layout(conv.to(dev)), g.to(dev), be.to(dev))
    torch.cuda.synchronize()
    assert torch.allclose(mean, mean2.cpu(), rtol=1e-5, atol=1e-6)
    assert torch.allclose(var, var2.cpu(), rtol=1e-5, atol=1e-6)
    diff = (out.float() - out2.cpu().float()).abs()
    assert diff.max().item() <= 2 ** -6 * max(1.0, out2.float().abs().max().item())


@pytest.mark.parametrize("stats", ["epilogue", "pass"])
def test_fused_is_deterministic(stats):
    say(f"fused determinism, stats={stats}")
    case = (4, 32, 64, 14, 14, 3, 1, 1, True, "bf16")
    x, w, b, g, be = _case(case, seed=11)
    r1 = _gpu(x, w, b, g, be, 1, 1, True, stats)
    r2 = _gpu(x, w, b, g, be, 1, 1, True, stats)
    for a, c in zip(r1, r2):
        assert torch.equal(a, c)


def _check_layer_statistics(xg, wg, g, be, stride, pad, label, stats="epilogue"):
    """mean/var of the fused call against fp64 statistics of the GPU
    convolution output, plus a sample of normalised values."""
    dev = torch.device("cuda:0")
    packed = quan.quan_qconv2d_pack_weights(*wg)
    shape = tuple(wg[0].shape)
    conv = quan.quan_qconv2d_forward_packed(xg, packed, shape, stride=stride, pad=pad)
    out, mean, var = quan.quan_qconv2d_iqbn_forward(xg, packed, shape, g, be, stride=stride, pad=pad,
                                                     stats=stats)
    torch.cuda.synchronize()
    c64 = conv.double()  # [N, 4, C, H, W] view of the device tensor, upcast on the GPU
    ref_mean = c64.mean(dim=(0, 3, 4))
    ref_var = ((c64 - ref_mean[None, :, :, None, None]) ** 2).mean(dim=(0, 3, 4))
    assert torch.allclose(mean.double(), ref_mean, rtol=1e-5, atol=1e-6), label
    assert torch.allclose(var.double(), ref_var, rtol=1e-5, atol=1e-6), label
    scale = g.double() / torch.sqrt(ref_var + 1e-5)
    ref = (c64 - ref_mean[None, :, :, None, None]) * scale[None, :, :, None, None] + be.double()[None, :, :, None, None]
    idx = torch.randint(0, out.numel(), (4096,), generator=torch.Generator().manual_seed(0)).to(dev)
    got = out.double().reshape(-1)[idx]
    exp = ref.reshape(-1)[idx]
    assert torch.all((got - exp).abs() <= 1e-2 + 2e-2 * exp.abs()), label


@pytest.mark.parametrize("stats", ["epilogue", "pass"])
def test_fused_statistics_at_full_layer_size(stats):
    """The imagenet_stage layer (64x56x56, 64->64): 1568 pixel tiles over the
    persistent work-groups, several tiles each."""
    say(f"fused full-size statistics, stats={stats}")
    from paper_2509_05512_amd import workloads
    wl = workloads.WORKLOADS["imagenet_stage"]
    tens = workloads.generate(wl)
    layer = tens.layers[0]
    dev = torch.device("cuda:0")
    xg = quan.to_device_layout(tens.x.to(dev))
    wg = [layer.weight[q].contiguous().to(dev) for q in range(4)]
    _check_layer_statistics(xg, wg, layer.gamma.to(dev), layer.beta.to(dev), 1, 1, "imagenet_stage", stats)


# (N, Cin, Cout, H, W, k): more pixel tiles than work-groups (each
# work-group gathers several tiles); ragged last tile.
MANY_TILES = [
    (8, 32, 64, 99, 101, 1),  # two stages per tile
    (4, 8, 32, 75, 77, 3),    # nine stages, 32-channel tiles
]


@pytest.mark.parametrize("case", MANY_TILES, ids=[str(c) for c in MANY_TILES])
def test_fused_statistics_many_tiles_per_work_group(case):
    say(f"fused statistics, many tiles {case}")
    N, Cin, Cout, H, W, k = case
    dev = torch.device("cuda:0")
    gen = torch.Generator(device="cpu").manual_seed(N * 1000 + Cin)
    x = torch.randn((N, 4, Cin, H, W), generator=gen).to(torch.bfloat16)
    w = (torch.randn((4, Cout, Cin, k, k), generator=gen) / (4 * Cin * k * k) ** 0.5).to(torch.bfloat16)
    g = torch.rand((4, Cout), generator=gen) + 0.5
    be = torch.randn((4, Cout), generator=gen) * 0.2
    xg = quan.to_device_layout(x.to(dev))
    wg = [w[q].contiguous().to(dev) for q in range(4)]
    _check_layer_statistics(xg, wg, g.to(dev), be.to(dev), 1, k // 2, str(case))


# ------------------------- inference IQBN folded in -------------------------

def _running_stats(case, seed):
    Cout = case[2]
    rng = np.random.default_rng(seed)
    rm = torch.from_numpy((rng.standard_normal((4, Cout)) * 0.5).astype(np.float32))
    rv = torch.from_numpy(rng.uniform(0.5, 2.0, (4, Cout)).astype(np.float32))
    return rm, rv


@pytest.mark.parametrize("relu", [False, True])
@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_inference_conv_iqbn_matches_oracle(case, relu):
    """quan_qconv2d_iqbn_inference against the oracle's conv followed by its
    inference IQBN (fp64), with random stored statistics."""
    say(f"inference conv+iqbn {case} relu={relu}")
    N, Cin, Cout, H, W, k, s, p, _, dtype = case
    dt = DT[dtype]
    seed = sum(map(ord, str(case))) % 997
    x, w, b, g, be = _case(case, seed=seed)
    rm, rv = _running_stats(case, seed + 1)
    dev = torch.device("cuda:0")
    xg = quan.to_device_layout(x.to(dev))
    wg = [w[q].contiguous().to(dev) for q in range(4)]
    packed = quan.quan_qconv2d_pack_weights(*wg)
    out = quan.quan_qconv2d_iqbn_inference(xg, packed, tuple(wg[0].shape), rm.to(dev), rv.to(dev), g.to(dev),
                                           be.to(dev), bias=b.to(dev), stride=s, pad=p, relu=relu)
    torch.cuda.synchronize()
    ref = oracle.iqbn_inference(oracle.qconv2d(f64(x), f64(w), f64(b), s, p, 1), f64(rm), f64(rv),
                                f64(g), f64(be), 1e-5, relu)
    assert_close(f64(out.cpu()), ref, dt, f"inference {case} relu={relu}")


def test_inference_with_batch_statistics_equals_training():
    """Stored statistics equal to the batch's own give the training-mode
    result (same conv output, same normalization up to rounding)."""
    say("inference vs training")
    case = (2, 32, 64, 14, 14, 3, 1, 1, True, "bf16")
    x, w, b, g, be = _case(case, seed=5)
    dev = torch.device("cuda:0")
    conv, out, mean, var = _gpu(x, w, b, g, be, 1, 1, True, "pass")
    xg = quan.to_device_layout(x.to(dev))
    wg = [w[q].contiguous().to(dev) for q in range(4)]
    packed = quan.quan_qconv2d_pack_weights(*wg)
    inf = quan.quan_qconv2d_iqbn_inference(xg, packed, tuple(wg[0].shape), mean.to(dev), var.to(dev),
                                           g.to(dev), be.to(dev), bias=b.to(dev), stride=1, pad=1, relu=True)
    torch.cuda.synchronize()
    # training normalizes the rounded conv output, inference the fp32
    # accumulator: one bf16 rounding apart
    assert_close(f64(inf.cpu()), f64(out), torch.bfloat16, "inference vs training")
