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
from parity import assert_close, conv_reference_sampled, f64, sample_pixels, say

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
    (2, 16, 64, 64, 64, 3, 1, 1, True, "bf16"),    # 256 statistics runs of 32 rows; pass: merged finalize
    (1, 16, 64, 65, 63, 3, 1, 1, False, "bf16"),   # 4095 rows: a ragged last statistics run
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


def _layer_inputs(case, seed):
    """Inputs of a large layer case (N, Cin, Cout, H, W, k): N(0,1)
    activations, N(0, 1/fan_in) kernels, a bias, gamma ~ U(0.5, 1.5), beta
    ~ N(0, 0.2^2), all rounded to bf16 / fp32 as the GPU receives them."""
    N, Cin, Cout, H, W, k = case
    rng = np.random.default_rng(seed)
    x = torch.from_numpy(rng.standard_normal((N, 4, Cin, H, W), dtype=np.float32)).to(torch.bfloat16)
    w = torch.from_numpy(rng.standard_normal((4, Cout, Cin, k, k), dtype=np.float32)
                         / np.float32(np.sqrt(4 * Cin * k * k))).to(torch.bfloat16)
    b = torch.from_numpy(rng.standard_normal((4, Cout), dtype=np.float32) * np.float32(0.3)).to(torch.bfloat16)
    g = torch.from_numpy(rng.uniform(0.5, 1.5, (4, Cout)).astype(np.float32))
    be = torch.from_numpy((rng.standard_normal((4, Cout)) * 0.2).astype(np.float32))
    return x, w, b, g, be


def _check_conv(x64, w64, b64, conv, stride, pad, k, label, full):
    """The GPU convolution output against the oracle convolution: in full, or
    (large layers) on sampled output pixels, all channels."""
    if full:
        assert_close(f64(conv), oracle.qconv2d(x64, w64, b64, stride, pad, 1), torch.bfloat16, f"conv {label}")
        return
    N, _, _, Ho, Wo = conv.shape
    rng = np.random.default_rng(3)
    picks = sample_pixels(rng, N, Ho, Wo, 40)
    ref = conv_reference_sampled(x64, w64, b64, stride, pad, 1, k, picks)
    got = np.stack([f64(conv[n, :, :, oy, ox]) for (n, oy, ox) in picks])
    assert_close(got, ref, torch.bfloat16, f"conv {label} (sampled)")


def _check_layer_statistics(case, stride, pad, relu, stats, seed, full_conv):
    """quan_qconv2d_iqbn_forward on a layer with more pixel tiles than
    work-groups (each persistent work-group gathers several tiles): its conv
    output against the oracle convolution, and out / mean / var element by
    element against the oracle's IQBN of that GPU convolution output."""
    N, Cin, Cout, H, W, k = case
    label = f"{case} s={stride} relu={relu} stats={stats}"
    x, w, b, g, be = _layer_inputs(case, seed)
    conv, out, mean, var = _gpu(x, w, b, g, be, stride, pad, relu, stats)
    _check_conv(f64(x), f64(w), f64(b), conv, stride, pad, k, label, full_conv)
    ref_out, ref_mean, ref_var = oracle.iqbn(f64(conv), f64(g), f64(be), 1e-5, relu)
    assert_close(mean.double().numpy(), ref_mean, torch.float32, f"mean {label}")
    assert_close(var.double().numpy(), ref_var, torch.float32, f"var {label}")
    assert_close(f64(out), ref_out, torch.bfloat16, f"out {label}")


IMAGENET = (64, 64, 64, 56, 56, 3)   # the imagenet_stage layer: 1568 pixel tiles


@pytest.mark.parametrize("relu", [False, True])
@pytest.mark.parametrize("stats", ["epilogue", "pass"])
def test_fused_statistics_at_full_layer_size(stats, relu):
    """The imagenet_stage layer (64x56x56, 64->64) with a bias: 1568 pixel
    tiles over the persistent work-groups, six or seven each."""
    say(f"fused full-size statistics, stats={stats} relu={relu}")
    _check_layer_statistics(IMAGENET, 1, 1, relu, stats, seed=21 + relu, full_conv=False)


# (N, Cin, Cout, H, W, k): more pixel tiles than work-groups (each
# work-group gathers several tiles); ragged last tile.
MANY_TILES = [
    (8, 32, 64, 99, 101, 1),  # 625 tiles, two stages per tile
    (4, 8, 32, 75, 77, 3),    # nine stages, 32-channel tiles
    (4, 32, 128, 45, 47, 3),  # two output-channel tiles, 18 stages
]


@pytest.mark.parametrize("relu", [False, True])
@pytest.mark.parametrize("stats", ["epilogue", "pass"])
@pytest.mark.parametrize("case", MANY_TILES, ids=[str(c) for c in MANY_TILES])
def test_fused_statistics_many_tiles_per_work_group(case, stats, relu):
    say(f"fused statistics, many tiles {case} stats={stats} relu={relu}")
    _check_layer_statistics(case, 1, case[5] // 2, relu, stats, seed=sum(case) + relu, full_conv=True)


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


def _fold_full(case, stride, pad, relu, seed, full_conv):
    """quan_qconv2d_iqbn_inference on a multi-tile layer against the oracle
    convolution followed by the oracle's inference IQBN: in full, or on
    sampled output pixels (each pixel's convolution from its own receptive
    field, then eq. 12 with the stored statistics)."""
    N, Cin, Cout, H, W, k = case
    label = f"{case} relu={relu}"
    x, w, b, g, be = _layer_inputs(case, seed)
    rm, rv = _running_stats((0, 0, Cout), seed + 1)
    dev = torch.device("cuda:0")
    xg = quan.to_device_layout(x.to(dev))
    wg = [w[q].contiguous().to(dev) for q in range(4)]
    packed = quan.quan_qconv2d_pack_weights(*wg)
    out = quan.quan_qconv2d_iqbn_inference(xg, packed, tuple(wg[0].shape), rm.to(dev), rv.to(dev), g.to(dev),
                                           be.to(dev), bias=b.to(dev), stride=stride, pad=pad, relu=relu)
    torch.cuda.synchronize()
    x64, w64, b64 = f64(x), f64(w), f64(b)
    if full_conv:
        ref = oracle.iqbn_inference(oracle.qconv2d(x64, w64, b64, stride, pad, 1), f64(rm), f64(rv), f64(g),
                                    f64(be), 1e-5, relu)
        assert_close(f64(out.cpu()), ref, torch.bfloat16, f"inference {label}")
        return
    Ho, Wo = out.shape[3], out.shape[4]
    rng = np.random.default_rng(seed)
    picks = sample_pixels(rng, N, Ho, Wo, 60)
    conv = conv_reference_sampled(x64, w64, b64, stride, pad, 1, k, picks)       # [S, 4, Cout]
    ref = oracle.iqbn_inference(conv[:, :, :, None, None], f64(rm), f64(rv), f64(g), f64(be), 1e-5, relu)
    got = np.stack([f64(out[n, :, :, oy, ox]) for (n, oy, ox) in picks])
    assert_close(got, ref[:, :, :, 0, 0], torch.bfloat16, f"inference {label} (sampled)")


@pytest.mark.parametrize("relu", [False, True])
def test_inference_full_layer_size(relu):
    """The folded epilogue at the imagenet_stage size the bench times."""
    say(f"inference full size relu={relu}")
    _fold_full(IMAGENET, 1, 1, relu, seed=31 + relu, full_conv=False)


@pytest.mark.parametrize("relu", [False, True])
@pytest.mark.parametrize("case", MANY_TILES, ids=[str(c) for c in MANY_TILES])
def test_inference_many_tiles_per_work_group(case, relu):
    say(f"inference many tiles {case} relu={relu}")
    _fold_full(case, 1, case[5] // 2, relu, seed=sum(case) + 2 * relu, full_conv=True)
