"""GPU parity of quan_poincare_map (Section III-A, eq. 4) through the C ABI
against the oracle's fp64 mapping, on seeded RGB images: ragged sizes, one
pixel, colours far outside the unit cube, and an ImageNet-sized batch."""
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
