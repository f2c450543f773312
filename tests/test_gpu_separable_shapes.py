"""More GPU parity cases of the separable form (eq. 7, bf16, stride 1),
each compared in full against the oracle: several tiles per work-group,
layers whose 128-pixel tiles cross image boundaries, 62-pixel rows, 14-pixel
rows, two output-channel tiles, a 5x5 kernel, no padding, three 32-channel
blocks, a 1x3 kernel, and a convolution without bias."""
import numpy as np
import pytest
import torch

import oracle
from paper_2509_05512_amd import quan
from parity import assert_close, f64, say

pytestmark = pytest.mark.gpu

BF16 = torch.bfloat16

# (N, Cin, Cout, H, W, k, pad) or (N, Cin, Cout, H, W, k_h, k_w, pad)
CASES = [
    (16, 64, 64, 56, 56, 3, 1),    # 392 tiles: two per work-group for some, tiles across images
    (4, 32, 64, 62, 62, 3, 1),     # 62-pixel rows, one 32-channel block
    (8, 64, 128, 14, 14, 3, 1),    # 14-pixel rows, two output-channel tiles
    (2, 32, 64, 20, 23, 5, 2),     # 5x5 kernel
    (3, 64, 64, 17, 19, 3, 0),     # no padding: 15 x 17 outputs
    (2, 96, 64, 11, 9, 3, 1),      # three channel blocks
    (2, 32, 64, 9, 12, 1, 3, 0),   # 1x3 kernel: three taps in one row
]


def _dims(case):
    if len(case) == 7:
        N, Cin, Cout, H, W, k, p = case
        return N, Cin, Cout, H, W, k, k, p
    return case


def _inputs(case, seed):
    N, Cin, Cout, H, W, kh, kw, _ = _dims(case)
    rng = np.random.default_rng(seed)
    x = torch.from_numpy(rng.standard_normal((N, 4, Cin, H, W), dtype=np.float32)).to(BF16)
    w = torch.from_numpy(rng.standard_normal((4, Cout, Cin, kh, kw), dtype=np.float32)
                         / np.float32(np.sqrt(Cin * kh * kw))).to(BF16)
    b = torch.from_numpy(rng.standard_normal((4, Cout), dtype=np.float32) * np.float32(0.3)).to(BF16)
    return x, w, b


@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_separable_shape_matches_oracle(case):
    say(f"separable shape {case}")
    N, Cin, Cout, H, W, kh, kw, p = _dims(case)
    x, w, b = _inputs(case, seed=sum(case))
    dev = torch.device("cuda:0")
    ho, wo = quan.conv_out_size(H, kh, 1, p, 1), quan.conv_out_size(W, kw, 1, p, 1)
    out = quan.empty_qmap(N, Cout, ho, wo, BF16, dev)
    out.fill_(float("nan"))
    quan.quan_qconv2d_separable_forward(quan.to_device_layout(x.to(dev)),
                                        *[w[q].contiguous().to(dev) for q in range(4)], bias=b.to(dev),
                                        stride=1, pad=p, out=out)
    torch.cuda.synchronize()
    ref = oracle.qconv2d_separable(f64(x), f64(w), f64(b), 1, p, 1)
    assert_close(f64(out), ref, BF16, f"separable shape {case}")


def test_separable_without_bias():
    case = (3, 64, 64, 17, 19, 3, 1)
    say(f"separable without bias {case}")
    N, Cin, Cout, H, W, k, p = case
    x, w, _ = _inputs(case, seed=5)
    dev = torch.device("cuda:0")
    out = quan.quan_qconv2d_separable_forward(quan.to_device_layout(x.to(dev)),
                                              *[w[q].contiguous().to(dev) for q in range(4)], stride=1, pad=p)
    torch.cuda.synchronize()
    assert_close(f64(out), oracle.qconv2d_separable(f64(x), f64(w), None, 1, p, 1), BF16, "separable no bias")
