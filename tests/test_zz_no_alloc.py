"""GPU check of quan_iqbn_forward_noalloc through the C ABI: two calls in a
row, the second on a smaller tensor, each equal to quan_iqbn_forward's
result (the same kernels on the same partial layout, so bit for bit) and to
the oracle within the bf16 bar; the scratch array keeps the first call's
partials, which the second call overwrites before it reads them."""
import numpy as np
import pytest
import torch

import oracle
from paper_2509_05512_amd import quan
from parity import assert_close, f64, say

pytestmark = pytest.mark.gpu


def _inputs(shape, seed):
    N, C, H, W = shape
    rng = np.random.default_rng(seed)
    x = torch.from_numpy((rng.standard_normal((N, 4, C, H, W)) * 1.3 + 0.4).astype(np.float32)).to(torch.bfloat16)
    g = torch.from_numpy(rng.uniform(0.5, 1.5, (4, C)).astype(np.float32))
    b = torch.from_numpy((rng.standard_normal((4, C)) * 0.2).astype(np.float32))
    return x, g, b


def _call(fn, x, g, b):
    dev = torch.device("cuda:0")
    xg = quan.to_device_layout(x.to(dev))
    n, _, c, h, w = x.shape
    out = quan.empty_qmap(n, c, h, w, x.dtype, dev).fill_(float("nan"))
    mean = torch.full((4, c), float("nan"), device=dev)
    var = torch.full((4, c), float("nan"), device=dev)
    fn(xg, g.to(dev), b.to(dev), 1e-5, out=out, mean=mean, var=var)
    torch.cuda.synchronize()
    return out.cpu(), mean.cpu(), var.cpu()


def test_noalloc_matches_workspace_entry_point_on_two_calls():
    for i, shape in enumerate([(16, 64, 28, 28), (2, 16, 9, 11)]):
        say(f"iqbn noalloc call {i} {shape}")
        x, g, b = _inputs(shape, seed=50 + i)
        got = _call(quan.quan_iqbn_forward_noalloc, x, g, b)
        ref = _call(quan.quan_iqbn_forward, x, g, b)
        for a, r, name in zip(got, ref, ("out", "mean", "var")):
            assert torch.equal(a, r), f"call {i}: {name} differs from quan_iqbn_forward"
        o_ref, m_ref, v_ref = oracle.iqbn(f64(x), f64(g), f64(b), 1e-5, False)
        assert_close(f64(got[1]), m_ref, torch.bfloat16, f"mean call {i}")
        assert_close(f64(got[2]), v_ref, torch.bfloat16, f"var call {i}")
        assert_close(f64(got[0]), o_ref, torch.bfloat16, f"out call {i}")
