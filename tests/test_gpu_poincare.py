"""GPU parity of quan_poincare_map (Section III-A, eq. 4) through the C ABI
against the oracle's fp64 mapping, on seeded RGB images: ragged sizes, one
pixel, colours far outside the unit cube, and an ImageNet-sized batch; and of
the stem convolution with the map fused into its loads
(quan_qconv2d_poincare_forward) against the oracle convolution of the
oracle map."""
import numpy as np
import pytest
import torch

import oracle
from paper_2509_05512_amd import quan
from parity import assert_close, f64, say

pytestmark = pytest.mark.gpu

DT = {"fp32": torch.float32, "bf16": torch.bfloat16}

# (N, H, W, scale of the colour values, dtype)
CASES = [
    (2, 17, 19, 1.0, "bf16"),     # plane of 323 pixels: one pixel per thread
    (2, 17, 19, 1.0, "fp32"),
    (3, 12, 20, 1.0, "bf16"),     # plane of 240 pixels: four per thread
    (3, 12, 20, 1.0, "fp32"),
    (2, 12, 21, 1.0, "bf16"),     # plane of 252 pixels (odd width): four per thread
    (2, 9, 30, 1.0, "fp32"),      # plane of 270 pixels: one per thread
    (1, 1, 1, 1.0, "bf16"),       # one pixel
    (3, 8, 33, 20.0, "fp32"),     # far outside the unit cube: q_r near -1
    (1, 5, 7, 0.0, "bf16"),       # black: q = 1
]


def _rgb(N, H, W, scale, dtype, seed):
    rng = np.random.default_rng(seed)
    return torch.from_numpy(rng.uniform(0.0, 1.0, (N, 3, H, W)).astype(np.float32) * np.float32(scale)).to(DT[dtype])


@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_poincare_matches_oracle(case):
    say(f"poincare {case}")
    N, H, W, scale, dtype = case
    rgb = _rgb(N, H, W, scale, dtype, seed=N * 100 + H)
    q = quan.quan_poincare_map(rgb.to("cuda:0"))
    torch.cuda.synchronize()
    got = f64(q.cpu())
    assert_close(got, oracle.poincare(f64(rgb)), DT[dtype], f"poincare {case}")
    if dtype == "fp32":
        assert np.allclose(np.linalg.norm(got, axis=1), 1.0, atol=2e-6), "unit norm"


def test_poincare_imagenet_batch():
    """64 x 3 x 224 x 224 (an ImageNet input batch), every pixel checked."""
    say("poincare imagenet batch")
    rgb = _rgb(64, 224, 224, 1.0, "bf16", seed=7)
    q = quan.quan_poincare_map(rgb.to("cuda:0"))
    torch.cuda.synchronize()
    assert_close(f64(q.cpu()), oracle.poincare(f64(rgb)), torch.bfloat16, "poincare imagenet")


def test_poincare_feeds_the_convolution():
    """The mapped image is a valid first-layer input: conv of the GPU map
    equals the oracle conv of the oracle map (within bf16 tolerance)."""
    say("poincare -> qconv2d")
    rgb = _rgb(2, 12, 10, 1.0, "bf16", seed=3)
    rng = np.random.default_rng(4)
    w = torch.from_numpy((rng.standard_normal((4, 32, 1, 3, 3)) / 6.0).astype(np.float32)).to(torch.bfloat16)
    dev = torch.device("cuda:0")
    q = quan.quan_poincare_map(rgb.to(dev))
    y = quan.quan_qconv2d_forward(q, *[w[p].contiguous().to(dev) for p in range(4)], stride=1, pad=1)
    torch.cuda.synchronize()
    # reference: the oracle conv of the GPU's (bf16) map, so only the conv's
    # own rounding is compared
    ref = oracle.qconv2d(f64(q.cpu()), f64(w), None, 1, 1, 1)
    assert_close(f64(y.cpu()), ref, torch.bfloat16, "poincare -> conv")


# ------------------- the Poincare map fused into the stem conv -------------------

# (N, H, W, Cout, k, stride, pad, colour scale, dtype)
STEM_CASES = [
    (2, 17, 19, 32, 3, 1, 1, 1.0, "bf16"),    # ragged planes and pixel tiles
    (2, 17, 19, 16, 3, 1, 1, 1.0, "fp32"),
    (3, 20, 22, 64, 3, 2, 1, 1.0, "bf16"),    # stride 2 (a detection stem), 64-channel tiles
    (2, 23, 21, 16, 7, 2, 3, 1.0, "bf16"),    # 7x7 stride 2 (a classification stem)
    (2, 9, 11, 12, 3, 1, 1, 1.0, "bf16"),     # 12 channels: not whole 16-byte output chunks
    (1, 8, 9, 32, 3, 1, 0, 15.0, "bf16"),     # colours far outside the unit cube
    # past the stem kernel's weight table: the implicit-GEMM kernel with the
    # map in its loads
    (2, 10, 12, 80, 3, 1, 1, 1.0, "bf16"),    # 80 channels: ten 32-row blocks
    (2, 13, 11, 64, 5, 1, 2, 1.0, "bf16"),    # 5x5, 64 channels: 8 x 7 fragments
]


def _stem(case, seed):
    N, H, W, Cout, k, s, p, scale, dtype = case
    dt = DT[dtype]
    rgb = _rgb(N, H, W, scale, dtype, seed)
    rng = np.random.default_rng(seed + 1)
    w = torch.from_numpy((rng.standard_normal((4, Cout, 1, k, k)) / np.sqrt(4 * k * k)).astype(np.float32)).to(dt)
    b = torch.from_numpy((rng.standard_normal((4, Cout)) * 0.1).astype(np.float32)).to(dt)
    return rgb, w, b


def _stem_gpu(rgb, w, b, s, p):
    dev = torch.device("cuda:0")
    ws = [w[q].contiguous().to(dev) for q in range(4)]
    packed = quan.quan_qconv2d_pack_weights(*ws)
    shape = tuple(ws[0].shape)
    rgb_d, b_d = rgb.to(dev), b.to(dev)
    fused = quan.quan_qconv2d_poincare_forward(rgb_d, packed, shape, bias=b_d, stride=s, pad=p)
    two_pass = quan.quan_qconv2d_forward_packed(quan.quan_poincare_map(rgb_d), packed, shape, bias=b_d, stride=s,
                                                pad=p)
    torch.cuda.synchronize()
    return fused.cpu(), two_pass.cpu()


@pytest.mark.parametrize("case", STEM_CASES, ids=[str(c) for c in STEM_CASES])
def test_fused_stem_matches_oracle(case):
    """The fused stem equals the oracle convolution of the oracle's fp64
    Poincare map (the GPU rounds each input quaternion once to dtype, as the
    separate map does), and the two-pass GPU path computes the same."""
    say(f"fused poincare stem {case}")
    N, H, W, Cout, k, s, p, scale, dtype = case
    dt = DT[dtype]
    rgb, w, b = _stem(case, seed=N * 31 + H)
    fused, two_pass = _stem_gpu(rgb, w, b, s, p)
    ref = oracle.qconv2d(oracle.poincare(f64(rgb)), f64(w), f64(b), s, p, 1)
    assert_close(f64(fused), ref, dt, f"fused stem {case}")
    assert_close(f64(fused), f64(two_pass), dt, f"fused vs two-pass {case}")


def test_fused_stem_imagenet_batch():
    """64 x 3 x 224 x 224 through a 3x3 stride-2 stem of 16 quaternion
    channels: the fused output against the oracle on sampled output pixels
    (each from its own receptive field) and against the two-pass GPU path in
    full."""
    say("fused poincare stem, imagenet batch")
    from parity import conv_reference_sampled, sample_pixels
    case = (64, 224, 224, 16, 3, 2, 1, 1.0, "bf16")
    N, H, W, Cout, k, s, p, _, _ = case
    rgb, w, b = _stem(case, seed=11)
    fused, two_pass = _stem_gpu(rgb, w, b, s, p)
    assert_close(f64(fused), f64(two_pass), torch.bfloat16, "fused vs two-pass, imagenet")
    ho, wo = fused.shape[3], fused.shape[4]
    picks = sample_pixels(np.random.default_rng(12), N, ho, wo, 48)
    q64 = oracle.poincare(f64(rgb))
    ref = conv_reference_sampled(q64, f64(w), f64(b), s, p, 1, k, picks)
    got = np.stack([f64(fused[n, :, :, oy, ox]) for (n, oy, ox) in picks])
    assert_close(got, ref, torch.bfloat16, "fused stem imagenet (sampled)")
