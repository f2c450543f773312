"""The five benchmark workloads end to end on the GPU, stage by stage against
the oracle, in the launch configuration the benchmark times.

The tiny fp32 layer is compared in full.  For the full-size bf16 layers the
convolution is compared on sampled output pixels (every channel of each; the
oracle evaluates each pixel on its own receptive field, corners and the last
pixel always included), and IQBN in full on the GPU's own convolution output,
so each stage's error is measured on its own."""
import numpy as np
import pytest
import torch

import oracle
from paper_2509_05512_amd import quan, workloads
from parity import assert_close, conv_reference_sampled, f64, sample_pixels, say

pytestmark = pytest.mark.gpu

SAMPLES = {"tiny_fp32": None, "cifar": 96, "imagenet_stage": 48, "detection_pair": 48,
           "deep_stack": 24}


@pytest.mark.parametrize("name", workloads.WORKLOAD_ORDER)
def test_workload_stages_match_oracle(name):
    wl = workloads.WORKLOADS[name]
    say(f"workload {name}: generating")
    tens = workloads.generate(wl)
    dev = torch.device("cuda:0")
    dt = wl.torch_dtype
    rng = np.random.default_rng(1234)
    x_gpu = quan.to_device_layout(tens.x.to(dev))
    for li, (L, lt) in enumerate(zip(wl.layers, tens.layers)):
        say(f"workload {name} layer {li}: conv {L}")
        w = [lt.weight[q].contiguous().to(dev) for q in range(4)]
        b = lt.bias.contiguous().to(dev) if lt.bias is not None else None
        y = quan.quan_qconv2d_forward(x_gpu, *w, bias=b, stride=L.stride, pad=L.pad,
                                      dilation=L.dilation)
        torch.cuda.synchronize()
        x64 = f64(x_gpu)
        w64 = f64(lt.weight)
        b64 = f64(lt.bias) if lt.bias is not None else None
        y64 = f64(y)
        if SAMPLES[name] is None:
            ref = oracle.qconv2d(x64, w64, b64, L.stride, L.pad, L.dilation)
            assert_close(y64, ref, dt, f"{name} layer {li} conv")
        else:
            N, _, _, ho, wo = y64.shape
            pix = sample_pixels(rng, N, ho, wo, SAMPLES[name])
            ref = conv_reference_sampled(x64, w64, b64, L.stride, L.pad, L.dilation, L.k, pix)
            got = np.stack([y64[n, :, :, oy, ox] for (n, oy, ox) in pix])
            assert_close(got, ref, dt, f"{name} layer {li} conv (sampled)")
        del x64
        say(f"workload {name} layer {li}: iqbn relu={L.relu}")
        g, be = lt.gamma.to(dev), lt.beta.to(dev)
        fn = quan.quan_iqbn_relu_forward if L.relu else quan.quan_iqbn_forward
        z, mean, var = fn(y, g, be, wl.eps)
        torch.cuda.synchronize()
        rz, rmean, rvar = oracle.iqbn(y64, f64(lt.gamma), f64(lt.beta), wl.eps, L.relu)
        assert_close(f64(mean), rmean, dt, f"{name} layer {li} mean")
        assert_close(f64(var), rvar, dt, f"{name} layer {li} var")
        assert_close(f64(z), rz, dt, f"{name} layer {li} iqbn out")
        x_gpu = z
    say(f"workload {name}: ok")
