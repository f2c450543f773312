"""GPU parity of the all-components convolution kernel on layers whose last
round of 128-pixel tiles would leave work-groups idle: those layers end in
32-pixel tail blocks, which the work-groups claim (one each, through a
per-stream counter) as they finish their tiles, each wave computing one
output component of the block, two K-blocks per ring slot.  With 256
compute units (one work-group each) a layer takes tail blocks when it runs
on the 64-channel tile with DMA loads (33..64 output channels, input
channels a multiple of 8 in bf16), its 32-pixel blocks number at least
4 x 256 and leave a remainder of 1..256 past a whole number of rounds, and
each work-group's tiles hold at least 8 K steps; the cases below are sized
for that, except those marked as whole tiles (on another device they are
all plain parity cases).

Every case is compared in full against the oracle: the bias epilogue (64-
and 32-channel tiles, a channel count without whole 16-byte output chunks,
one tail block, a tail block for every work-group, two full rounds before
the tail, stride 2, and a 1x1 layer, which the pointwise kernel takes), the
IQBN statistics gathered in the epilogue with a ragged last block, the
folded inference epilogue, and the Poincare stem with the map in the
kernel's loads."""
import numpy as np
import pytest
import torch

import oracle
from paper_2509_05512_amd import quan
from parity import assert_close, f64, say

pytestmark = pytest.mark.gpu

BF16 = torch.bfloat16


def tail_blocks(pixels, steps, work_groups=256):
    """Tail blocks the launch takes for a layer of `pixels` output pixels and
    `steps` K steps per tile on the 64-channel DMA tile (the host's rule),
    for the case labels."""
    blk = -(-pixels // 32)
    full = blk // (4 * work_groups)
    rest = blk - 4 * work_groups * full
    return rest if full >= 1 and 0 < rest <= work_groups and full * steps >= 8 else 0


# (N, Cin, Cout, H, W, k, stride, pad)
CONV_CASES = [
    (8, 16, 64, 66, 66, 3, 1, 1),     # 1089 blocks: 65 tail blocks, nine K steps (odd: last step one K-block)
    (8, 16, 32, 66, 66, 3, 1, 1),     # 32-channel tile: whole tiles
    (8, 16, 36, 66, 66, 3, 1, 1),     # c_out % 8 != 0: direct stores
    (8, 8, 64, 41, 100, 3, 1, 1),     # 1025 blocks: one tail block
    (8, 16, 64, 64, 80, 3, 1, 1),     # 1280 blocks: a tail block per work-group
    (8, 64, 64, 64, 80, 1, 1, 0),     # 1x1: the pointwise streaming kernel (no tail blocks)
    (8, 16, 64, 92, 92, 3, 1, 1),     # 2116 blocks: two full rounds, 68 tail blocks
    (8, 16, 64, 131, 131, 3, 2, 1),   # stride 2 to 66 x 66
    (8, 16, 64, 65, 67, 3, 1, 1),     # 34840 pixels: ragged last tail block
    (8, 32, 64, 66, 66, 3, 1, 1),     # 18 K steps (even)
]


def _inputs(case, seed):
    N, Cin, Cout, H, W, k = case[:6]
    rng = np.random.default_rng(seed)
    x = torch.from_numpy(rng.standard_normal((N, 4, Cin, H, W), dtype=np.float32)).to(BF16)
    w = torch.from_numpy(rng.standard_normal((4, Cout, Cin, k, k), dtype=np.float32)
                         / np.float32(np.sqrt(4 * Cin * k * k))).to(BF16)
    b = torch.from_numpy(rng.standard_normal((4, Cout), dtype=np.float32) * np.float32(0.3)).to(BF16)
    return x, w, b


def _label(case):
    N, Cin, Cout, H, W, k, s, p = case
    ho, wo = quan.conv_out_size(H, k, s, p, 1), quan.conv_out_size(W, k, s, p, 1)
    steps = k * k * -(-Cin // 16)
    dma_64 = 32 < Cout <= 64 and Cin % 8 == 0
    return f"{case} tail_blocks={tail_blocks(N * ho * wo, steps) if dma_64 else 0}"


@pytest.mark.parametrize("case", CONV_CASES, ids=[str(c) for c in CONV_CASES])
def test_tail_blocks_conv_matches_oracle(case):
    label = _label(case)
    say(f"tail blocks conv {label}")
    N, Cin, Cout, H, W, k, s, p = case
    x, w, b = _inputs(case, seed=sum(case))
    dev = torch.device("cuda:0")
    ho, wo = quan.conv_out_size(H, k, s, p, 1), quan.conv_out_size(W, k, s, p, 1)
    out = quan.empty_qmap(N, Cout, ho, wo, BF16, dev)
    out.fill_(float("nan"))
    quan.quan_qconv2d_forward(quan.to_device_layout(x.to(dev)), *[w[q].contiguous().to(dev) for q in range(4)],
                              bias=b.to(dev), stride=s, pad=p, out=out)
    torch.cuda.synchronize()
    assert_close(f64(out), oracle.qconv2d(f64(x), f64(w), f64(b), s, p, 1), BF16, f"tail conv {label}")


@pytest.mark.parametrize("relu", [False, True])
@pytest.mark.parametrize("stats", ["epilogue", "pass"])
def test_tail_blocks_statistics(stats, relu):
    """Convolution + IQBN with a ragged last tail block: the conv output
    against the oracle convolution, and out / mean / var against the
    oracle's IQBN of that GPU conv output."""
    case = (8, 16, 64, 65, 67, 3, 1, 1)
    label = f"{_label(case)} stats={stats} relu={relu}"
    say(f"tail blocks statistics {label}")
    N, Cin, Cout, H, W, k, s, p = case
    x, w, b = _inputs(case, seed=77 + relu)
    rng = np.random.default_rng(78)
    g = torch.from_numpy(rng.uniform(0.5, 1.5, (4, Cout)).astype(np.float32))
    be = torch.from_numpy((rng.standard_normal((4, Cout)) * 0.2).astype(np.float32))
    dev = torch.device("cuda:0")
    xg = quan.to_device_layout(x.to(dev))
    wg = [w[q].contiguous().to(dev) for q in range(4)]
    packed = quan.quan_qconv2d_pack_weights(*wg)
    shape = tuple(wg[0].shape)
    conv = quan.quan_qconv2d_forward_packed(xg, packed, shape, bias=b.to(dev), stride=s, pad=p)
    out, mean, var = quan.quan_qconv2d_iqbn_forward(xg, packed, shape, g.to(dev), be.to(dev), bias=b.to(dev),
                                                     stride=s, pad=p, relu=relu, stats=stats)
    torch.cuda.synchronize()
    conv, out, mean, var = conv.cpu(), out.cpu(), mean.cpu(), var.cpu()
    assert_close(f64(conv), oracle.qconv2d(f64(x), f64(w), f64(b), s, p, 1), BF16, f"tail conv {label}")
    ref_out, ref_mean, ref_var = oracle.iqbn(f64(conv), f64(g), f64(be), 1e-5, relu)
    assert_close(mean.double().numpy(), ref_mean, torch.float32, f"mean {label}")
    assert_close(var.double().numpy(), ref_var, torch.float32, f"var {label}")
    assert_close(f64(out), ref_out, BF16, f"out {label}")


@pytest.mark.parametrize("relu", [False, True])
def test_tail_blocks_inference(relu):
    """The folded inference epilogue (stored statistics, eq. 12) on tail
    blocks."""
    case = (8, 16, 64, 65, 67, 3, 1, 1)
    label = f"{_label(case)} relu={relu}"
    say(f"tail blocks inference {label}")
    N, Cin, Cout, H, W, k, s, p = case
    x, w, b = _inputs(case, seed=91 + relu)
    rng = np.random.default_rng(92)
    g = torch.from_numpy(rng.uniform(0.5, 1.5, (4, Cout)).astype(np.float32))
    be = torch.from_numpy((rng.standard_normal((4, Cout)) * 0.2).astype(np.float32))
    rm = torch.from_numpy((rng.standard_normal((4, Cout)) * 0.5).astype(np.float32))
    rv = torch.from_numpy(rng.uniform(0.5, 2.0, (4, Cout)).astype(np.float32))
    dev = torch.device("cuda:0")
    wg = [w[q].contiguous().to(dev) for q in range(4)]
    packed = quan.quan_qconv2d_pack_weights(*wg)
    out = quan.quan_qconv2d_iqbn_inference(quan.to_device_layout(x.to(dev)), packed, tuple(wg[0].shape),
                                           rm.to(dev), rv.to(dev), g.to(dev), be.to(dev), bias=b.to(dev),
                                           stride=s, pad=p, relu=relu)
    torch.cuda.synchronize()
    ref = oracle.iqbn_inference(oracle.qconv2d(f64(x), f64(w), f64(b), s, p, 1), f64(rm), f64(rv), f64(g),
                                f64(be), 1e-5, relu)
    assert_close(f64(out.cpu()), ref, BF16, f"tail inference {label}")


def test_tail_blocks_poincare_stem():
    """A 5x5 stem of 64 quaternion channels (past the dedicated stem
    kernel's weight table, so the implicit-GEMM kernel with the map of eq. 4
    in its loads runs it) on 8 images of 66 x 66, a size with a partial last
    round: the stem variant (element loads) runs whole tiles."""
    N, H, W, Cout, k, p = 8, 66, 66, 64, 5, 2
    say("tail-sized poincare stem")
    rng = np.random.default_rng(5)
    rgb = torch.from_numpy(rng.uniform(0.0, 1.0, (N, 3, H, W)).astype(np.float32)).to(BF16)
    w = torch.from_numpy((rng.standard_normal((4, Cout, 1, k, k)) / np.sqrt(4 * k * k)).astype(np.float32)).to(BF16)
    b = torch.from_numpy((rng.standard_normal((4, Cout)) * 0.1).astype(np.float32)).to(BF16)
    dev = torch.device("cuda:0")
    ws = [w[q].contiguous().to(dev) for q in range(4)]
    packed = quan.quan_qconv2d_pack_weights(*ws)
    out = quan.quan_qconv2d_poincare_forward(rgb.to(dev), packed, tuple(ws[0].shape), bias=b.to(dev), stride=1,
                                             pad=p)
    torch.cuda.synchronize()
    ref = oracle.qconv2d(oracle.poincare(f64(rgb)), f64(w), f64(b), 1, p, 1)
    assert_close(f64(out.cpu()), ref, BF16, "tail poincare stem")


def _tail_conv(x, w, b, s, p, stream=None):
    dev = torch.device("cuda:0")
    N, _, Cin, H, W = x.shape
    Cout, k = w.shape[1], w.shape[3]
    ho, wo = quan.conv_out_size(H, k, s, p, 1), quan.conv_out_size(W, k, s, p, 1)
    out = quan.empty_qmap(N, Cout, ho, wo, BF16, dev)
    out.fill_(float("nan"))
    quan.quan_qconv2d_forward(quan.to_device_layout(x.to(dev)), *[w[q].contiguous().to(dev) for q in range(4)],
                              bias=b.to(dev), stride=s, pad=p, out=out)
    return out


def test_tail_blocks_repeated_launches():
    """Back-to-back launches on one stream share its claim counter, which
    each launch must leave at zero: three launches of one layer and one of
    another, each into NaN-filled outputs, all equal to the oracle."""
    say("tail blocks repeated launches")
    cases = [(8, 16, 64, 66, 66, 3, 1, 1)] * 3 + [(8, 8, 64, 41, 100, 3, 1, 1)]
    outs = []
    for i, case in enumerate(cases):
        x, w, b = _inputs(case, seed=500 + (i if i == 3 else 0))
        outs.append((case, x, w, b, _tail_conv(x, w, b, case[6], case[7])))
    torch.cuda.synchronize()
    refs = {}
    for case, x, w, b, out in outs:
        if case not in refs:
            refs[case] = oracle.qconv2d(f64(x), f64(w), f64(b), case[6], case[7], 1)
        assert_close(f64(out.cpu()), refs[case], BF16, f"repeated tail conv {_label(case)}")


def test_tail_blocks_two_streams():
    """Two layers with tail blocks launched on two streams without a sync
    between them (each stream has its own claim counter), then a third on
    the first stream again."""
    say("tail blocks on two streams")
    dev = torch.device("cuda:0")
    c1, c2 = (8, 16, 64, 66, 66, 3, 1, 1), (8, 16, 32, 66, 66, 3, 1, 1)
    i1, i2 = _inputs(c1, seed=601), _inputs(c2, seed=602)
    s1, s2 = torch.cuda.Stream(device=dev), torch.cuda.Stream(device=dev)
    torch.cuda.synchronize()
    with torch.cuda.stream(s1):
        o1 = _tail_conv(*i1, 1, 1)
    with torch.cuda.stream(s2):
        o2 = _tail_conv(*i2, 1, 1)
    with torch.cuda.stream(s1):
        o3 = _tail_conv(*i1, 1, 1)
    torch.cuda.synchronize()
    r1 = oracle.qconv2d(f64(i1[0]), f64(i1[1]), f64(i1[2]), 1, 1, 1)
    r2 = oracle.qconv2d(f64(i2[0]), f64(i2[1]), f64(i2[2]), 1, 1, 1)
    assert_close(f64(o1.cpu()), r1, BF16, "stream 1, first")
    assert_close(f64(o2.cpu()), r2, BF16, "stream 2")
    assert_close(f64(o3.cpu()), r1, BF16, "stream 1, second")


# (N, Cin, Cout, H, W, k, stride, pad) of the forward layer: input gradients
# whose stride-1 convolutions (one per output phase of a strided layer) end
# in tail blocks
GRAD_CASES = [
    (8, 16, 64, 132, 132, 3, 2, 1),   # four phases of 8 x 66 x 66 pixels into 16 channels: whole tiles
    (8, 64, 32, 132, 132, 3, 2, 1),   # into 64 channels: the 2 x 2-tap phase (8 K steps) takes tail blocks
    (8, 64, 16, 66, 66, 3, 1, 1),     # stride 1: one gradient convolution of 34848 pixels, tail blocks
]


@pytest.mark.parametrize("case", GRAD_CASES, ids=[str(c) for c in GRAD_CASES])
def test_tail_blocks_input_gradient(case):
    """quan_qconv2d_backward_data on layers whose gradient convolutions take
    tail blocks, against the oracle's input gradient in full."""
    N, Cin, Cout, H, W, k, s, p = case
    say(f"tail blocks input gradient {case}")
    rng = np.random.default_rng(sum(case))
    Ho, Wo = quan.conv_out_size(H, k, s, p, 1), quan.conv_out_size(W, k, s, p, 1)
    w = torch.from_numpy(rng.standard_normal((4, Cout, Cin, k, k), dtype=np.float32)
                         / np.float32(np.sqrt(4 * Cin * k * k))).to(BF16)
    dy = torch.from_numpy(rng.standard_normal((N, 4, Cout, Ho, Wo), dtype=np.float32)).to(BF16)
    dev = torch.device("cuda:0")
    dx = quan.empty_qmap(N, Cin, H, W, BF16, dev)
    dx.fill_(float("nan"))
    quan.quan_qconv2d_backward_data(quan.to_device_layout(dy.to(dev)), *[w[q].contiguous().to(dev) for q in range(4)],
                                    (H, W), stride=s, pad=p, dx=dx)
    torch.cuda.synchronize()
    x0 = np.zeros((N, 4, Cin, H, W))
    ref, _, _ = oracle.qconv2d_backward(x0, f64(w), f64(dy), s, p, 1)
    assert_close(f64(dx.cpu()), ref, BF16, f"tail dX {case}")
