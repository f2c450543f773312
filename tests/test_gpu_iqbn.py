"""GPU parity of quan_iqbn_forward / quan_iqbn_relu_forward against the CPU
oracle, through the C ABI: statistics and normalised output, both dtypes,
vector and scalar column paths, in-place use and the degenerate cases."""
import numpy as np
import pytest
import torch

import oracle
from paper_2509_05512_amd import quan
from parity import assert_close, f64, say

pytestmark = pytest.mark.gpu

DT = {"fp32": torch.float32, "bf16": torch.bfloat16}

# (N, C, H, W)
SHAPES = [
    (2, 4, 16, 16),        # the tiny layer
    (3, 16, 7, 9),
    (1, 64, 13, 11),
    (5, 3, 5, 5),          # 4C = 12: scalar column path for bf16
    (2, 256, 3, 3),        # wide rows
    (1, 600, 2, 3),        # more than one column group
    (7, 2, 1, 1),
    (1, 1, 1, 1),          # one value per column
    (64, 8, 32, 16),       # many rows, many blocks
    (32, 256, 14, 14),     # the deep-stack layer
    (64, 16, 32, 32),      # 86 statistics blocks per column group
    (2, 65, 5, 7),         # 4C = 260: bf16 scalar columns in 64-column groups, a short last group
    (16, 64, 24, 20),      # 256 columns, 7680 rows: 8 row blocks of the merged normalization
]


def _case(shape, dtype, seed, shift=0.0):
    N, C, H, W = shape
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((N, 4, C, H, W), dtype=np.float32) * np.float32(1.7)
    x += np.float32(shift) + rng.standard_normal((1, 4, C, 1, 1), dtype=np.float32)
    g = rng.uniform(0.5, 1.5, (4, C)).astype(np.float32)
    b = (rng.standard_normal((4, C), dtype=np.float32) * np.float32(0.3))
    return torch.from_numpy(x).to(dtype), torch.from_numpy(g), torch.from_numpy(b)


def _run(x, g, b, eps, relu, inplace=False):
    dev = torch.device("cuda:0")
    xg = quan.to_device_layout(x.to(dev))
    gg, bg = g.to(dev), b.to(dev)
    out = xg if inplace else quan.empty_qmap(*x.shape[:1], x.shape[2], x.shape[3], x.shape[4],
                                              x.dtype, dev).fill_(float("nan"))
    mean = torch.full((4, x.shape[2]), float("nan"), device=dev)
    var = torch.full((4, x.shape[2]), float("nan"), device=dev)
    fn = quan.quan_iqbn_relu_forward if relu else quan.quan_iqbn_forward
    fn(xg, gg, bg, eps, out=out, mean=mean, var=var)
    torch.cuda.synchronize()
    return out, mean, var


@pytest.mark.parametrize("relu", [False, True])
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_iqbn_matches_oracle(shape, dtype, relu):
    say(f"iqbn parity {dtype} {shape} relu={relu}")
    dt = DT[dtype]
    x, g, b = _case(shape, dt, seed=sum(shape))
    out, mean, var = _run(x, g, b, 1e-5, relu)
    ref, rmean, rvar = oracle.iqbn(f64(x), f64(g), f64(b), 1e-5, relu)
    assert_close(f64(mean), rmean, dt, "mean")
    assert_close(f64(var), rvar, dt, "var")
    assert_close(f64(out), ref, dt, "out")


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_iqbn_large_offset_does_not_cancel(dtype):
    """|mean| >> std: the shifted accumulation keeps the variance accurate."""
    say(f"iqbn offset {dtype}")
    dt = DT[dtype]
    x, g, b = _case((4, 8, 12, 12), dt, seed=3, shift=300.0)
    out, mean, var = _run(x, g, b, 1e-5, False)
    ref, rmean, rvar = oracle.iqbn(f64(x), f64(g), f64(b), 1e-5, False)
    assert_close(f64(var), rvar, dt, "var")
    assert_close(f64(out), ref, dt, "out")


@pytest.mark.parametrize("shape", [(3, 16, 10, 10), (4, 96, 9, 10)], ids=str)
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_iqbn_in_place(dtype, shape):
    """In place, with the finalize in its own launch (16 channels) and merged
    into the normalization (96 channels: six 64-column groups)."""
    say(f"iqbn in-place {dtype} {shape}")
    dt = DT[dtype]
    x, g, b = _case(shape, dt, seed=4)
    out, mean, var = _run(x, g, b, 1e-5, True, inplace=True)
    ref, _, _ = oracle.iqbn(f64(x), f64(g), f64(b), 1e-5, True)
    assert_close(f64(out), ref, dt, "in-place out")


def test_iqbn_constant_input_gives_beta():
    say("iqbn constant input")
    x = torch.full((2, 4, 6, 5, 5), 3.25)
    g = torch.rand(4, 6) + 0.5
    b = torch.randn(4, 6)
    out, mean, var = _run(x, g, b, 1e-5, False)
    assert torch.all(var.cpu() == 0)
    assert torch.allclose(mean.cpu(), torch.full((4, 6), 3.25))
    assert torch.allclose(out.cpu(), b[None, :, :, None, None].expand(2, 4, 6, 5, 5), atol=1e-6)


@pytest.mark.parametrize("shape", [(16, 32, 14, 14), (16, 64, 14, 14)], ids=str)
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_iqbn_deterministic(dtype, shape):
    """Bit-identical across calls: three launches (128 columns) and the
    merged two launches (256 columns: every block of a column group merges
    the partials itself, in one fixed order)."""
    say(f"iqbn determinism {dtype} {shape}")
    dt = DT[dtype]
    x, g, b = _case(shape, dt, seed=8)
    o1, m1, v1 = _run(x, g, b, 1e-5, False)
    o2, m2, v2 = _run(x, g, b, 1e-5, False)
    assert torch.equal(o1.cpu(), o2.cpu()) and torch.equal(m1.cpu(), m2.cpu()) \
        and torch.equal(v1.cpu(), v2.cpu())


@pytest.mark.parametrize("case", [("bf16", True), ("fp32", False)])
def test_iqbn_two_column_groups_many_block_groups(case):
    """18432 rows of 2400 columns: two column groups of 512 statistics blocks
    each, merged per column in block order."""
    dtype, relu = case
    say(f"iqbn column groups x block groups {dtype} relu={relu}")
    dt = DT[dtype]
    x, g, b = _case((8, 600, 48, 48), dt, seed=21)
    out, mean, var = _run(x, g, b, 1e-5, relu)
    ref, rmean, rvar = oracle.iqbn(f64(x), f64(g), f64(b), 1e-5, relu)
    assert_close(f64(mean), rmean, dt, "mean")
    assert_close(f64(var), rvar, dt, "var")
    assert_close(f64(out), ref, dt, "out")


def test_iqbn_repeated_calls_reuse_counters():
    """Calls of different shapes one after another on one stream sharing one
    workspace: every call matches the oracle, and repeating a call repeats
    its result bit for bit."""
    say("iqbn repeated calls")
    shapes = [(64, 16, 32, 32), (32, 256, 14, 14), (64, 16, 32, 32), (2, 4, 16, 16), (64, 16, 32, 32)]
    first = None
    for i, shape in enumerate(shapes):
        x, g, b = _case(shape, torch.bfloat16, seed=40 + (i % 2))
        out, mean, var = _run(x, g, b, 1e-5, False)
        ref, rmean, rvar = oracle.iqbn(f64(x), f64(g), f64(b), 1e-5, False)
        assert_close(f64(var), rvar, torch.bfloat16, f"var call {i}")
        assert_close(f64(out), ref, torch.bfloat16, f"out call {i}")
        if shape == shapes[0]:
            if first is None:
                first = (out.cpu(), mean.cpu(), var.cpu())
            elif i == 4:
                assert torch.equal(first[0], out.cpu()) and torch.equal(first[2], var.cpu())


# ---- the one-launch form (tensors that fit the registers and LDS of one
# work-group per compute unit: above 32 MiB, or from 16 MiB where the rows
# span fewer than four 64-column groups) -------------------------------------

def _cus():
    return torch.cuda.get_device_properties(0).multi_processor_count


# (N, C, H, W), dtype, relu: narrow rows (8 chunks, 16 MiB), 512-byte and
# 1 KB rows (32 and 64 chunks), 4 KB and 8 KB rows (several columns merged
# per work-group), the detection-pair layer and the full ImageNet-stage layer
RESIDENT = [
    ((128, 16, 32, 32), "bf16", True),
    ((64, 64, 32, 32), "bf16", False),
    ((32, 64, 32, 32), "fp32", True),
    ((8, 512, 32, 32), "bf16", False),
    ((2, 1024, 32, 64), "bf16", True),
    ((16, 64, 80, 80), "bf16", False),
    ((64, 64, 56, 56), "bf16", True),
]


@pytest.mark.parametrize("shape,dtype,relu", RESIDENT, ids=[f"{s}-{d}-relu{int(r)}" for s, d, r in RESIDENT])
def test_iqbn_one_launch_matches_oracle(shape, dtype, relu):
    say(f"iqbn one-launch {dtype} {shape} relu={relu}")
    dt = DT[dtype]
    x, g, b = _case(shape, dt, seed=sum(shape) + 5)
    out, mean, var = _run(x, g, b, 1e-5, relu)
    ref, rmean, rvar = oracle.iqbn(f64(x), f64(g), f64(b), 1e-5, relu)
    assert_close(f64(mean), rmean, dt, "mean")
    assert_close(f64(var), rvar, dt, "var")
    assert_close(f64(out), ref, dt, "out")


# 16 MiB tensors with four or more 64-column groups: the merged two-launch
# form (statistics, then the finalize merged into the normalization)
MERGED = [
    ((32, 64, 32, 32), "bf16", False),
    ((16, 64, 32, 32), "fp32", True),
    ((4, 512, 32, 32), "bf16", True),
]


@pytest.mark.parametrize("shape,dtype,relu", MERGED, ids=[f"{s}-{d}-relu{int(r)}" for s, d, r in MERGED])
def test_iqbn_merged_16mib_matches_oracle(shape, dtype, relu):
    say(f"iqbn merged {dtype} {shape} relu={relu}")
    dt = DT[dtype]
    x, g, b = _case(shape, dt, seed=sum(shape) + 6)
    out, mean, var = _run(x, g, b, 1e-5, relu)
    ref, rmean, rvar = oracle.iqbn(f64(x), f64(g), f64(b), 1e-5, relu)
    assert_close(f64(mean), rmean, dt, "mean")
    assert_close(f64(var), rvar, dt, "var")
    assert_close(f64(out), ref, dt, "out")


@pytest.mark.parametrize("extra", [0, 16])
def test_iqbn_one_launch_capacity_edge(extra):
    """256-element bf16 rows: 16 rows per pass of a work-group, at most 51
    passes held per work-group.  The largest tensor held (51 passes on every
    compute unit) and one just past it (the three launches) both match."""
    P = _cus() * 16 * 51 + extra
    say(f"iqbn capacity edge P={P}")
    x, g, b = _case((1, 64, 1, P), torch.bfloat16, seed=77 + extra)
    out, mean, var = _run(x, g, b, 1e-5, False)
    ref, rmean, rvar = oracle.iqbn(f64(x), f64(g), f64(b), 1e-5, False)
    assert_close(f64(var), rvar, torch.bfloat16, "var")
    assert_close(f64(out), ref, torch.bfloat16, "out")


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_iqbn_one_launch_in_place_and_repeatable(dtype):
    """In place (every work-group reads all its rows before any is written),
    and bit-identical across calls (fixed-order merges; the barrier flags
    advance by two per call)."""
    say(f"iqbn one-launch in-place {dtype}")
    dt = DT[dtype]
    x, g, b = _case((64, 64, 32, 32), dt, seed=91)
    o1, m1, v1 = _run(x, g, b, 1e-5, True, inplace=True)
    ref, rmean, rvar = oracle.iqbn(f64(x), f64(g), f64(b), 1e-5, True)
    assert_close(f64(o1), ref, dt, "in-place out")
    for _ in range(3):
        o2, m2, v2 = _run(x, g, b, 1e-5, True, inplace=True)
        assert torch.equal(o1.cpu(), o2.cpu()) and torch.equal(m1.cpu(), m2.cpu()) \
            and torch.equal(v1.cpu(), v2.cpu())
