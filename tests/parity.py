"""Helpers for comparing the GPU path with the CPU oracle.

Tolerances (the bar every parity test applies):
  fp32: normwise  max|gpu - ref| <= 1e-5 * max|ref|
  bf16: elementwise |gpu - ref| <= 1e-2 + 2e-2 * |ref|
The reference is the fp64 oracle run on exactly the (rounded) values the GPU
received; it is never rounded itself."""
import numpy as np
import torch

import oracle

FP32_RTOL = 1e-5
BF16_ATOL, BF16_RTOL = 1e-2, 2e-2


def say(msg):
    print(msg, flush=True)


def f64(t: torch.Tensor) -> np.ndarray:
    """Logical-layout float64 copy of a (CPU or GPU) tensor."""
    return t.detach().to("cpu", torch.float64).numpy()


def assert_close(got, ref, dtype, what=""):
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite values in GPU output"
    err = np.abs(got - ref)
    if dtype == torch.float32:
        scale = float(np.max(np.abs(ref))) if ref.size else 0.0
        worst = float(err.max()) if err.size else 0.0
        assert worst <= FP32_RTOL * max(scale, 1e-30), \
            f"{what}: fp32 normwise error {worst:.3e} > 1e-5 * {scale:.3e}"
        return worst / max(scale, 1e-30)
    bound = BF16_ATOL + BF16_RTOL * np.abs(ref)
    bad = err > bound
    if bad.any():
        i = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError(f"{what}: {int(bad.sum())} of {err.size} outside bf16 tolerance; "
                             f"worst at {i}: got {got[i]:.6g} ref {ref[i]:.6g}")
    return float((err / (BF16_ATOL + BF16_RTOL * np.abs(ref))).max()) if err.size else 0.0


def conv_reference_sampled(x64, w64, b64, stride, pad, dil, k, samples, conv=None):
    """Oracle values at the sampled output pixels [(n, oy, ox), ...], all
    channels: each pixel is the oracle run on its own receptive field
    (conv: the oracle convolution to use, the Hamilton one by default)."""
    conv = conv or oracle.qconv2d
    N, _, Cin, H, W = x64.shape
    span = dil * (k - 1) + 1
    xp = np.pad(x64, ((0, 0), (0, 0), (0, 0), (pad, pad), (pad, pad)))
    patches = np.stack([xp[n, :, :, oy * stride:oy * stride + span, ox * stride:ox * stride + span]
                        for (n, oy, ox) in samples])
    y = conv(patches, w64, b64, stride=1, pad=0, dilation=dil)
    return y[:, :, :, 0, 0]                      # [S, 4, Cout]


def sample_pixels(rng, n, ho, wo, count):
    """Random output pixels, always including the four corners of the first
    and last images (padding edges) and the last pixel (ragged M tail)."""
    fixed = [(0, 0, 0), (0, 0, wo - 1), (0, ho - 1, 0), (n - 1, ho - 1, wo - 1),
             (n - 1, 0, wo - 1), (n - 1, ho - 1, 0)]
    picks = [(int(rng.integers(n)), int(rng.integers(ho)), int(rng.integers(wo)))
             for _ in range(count)]
    return list(dict.fromkeys(fixed + picks))
