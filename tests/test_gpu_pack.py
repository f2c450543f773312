"""GPU check of the weight pack (quan_qconv2d_pack_weights): pure data
movement, so the packed buffer must equal, bit for bit, the layout the
convolution kernels read, built here with numpy from its definition:
[tap][channel block][kernel r, i, j, k][output channel, padded to 64][16
input channels (bf16) or 8 (fp32)], zeros in the padding.

Cases: 3x3 and 1x1 kernels whose input channels come in whole octets from
16-byte aligned tensors (the octet kernel), a channel count that leaves half
a block and output padding, kernel sizes the octet kernel does not take, a
source that is only 2-byte aligned, and fp32 (the element kernel)."""
import numpy as np
import pytest
import torch

from paper_2509_05512_amd import quan
from parity import say

pytestmark = pytest.mark.gpu


def reference_pack(ws, dtype):
    """The packed layout from its definition (numpy, logical order)."""
    w = np.stack([t.cpu().contiguous().view(torch.int16 if dtype == torch.bfloat16 else torch.int32).numpy()
                  for t in ws])  # [4][Cout][Cin][kh][kw], raw bits
    _, c_out, c_in, k_h, k_w = w.shape
    pk = 16 if dtype == torch.bfloat16 else 8
    n_cblk = -(-c_in // pk)
    cout_pad = -(-c_out // 64) * 64
    out = np.zeros((k_h * k_w, n_cblk, 4, cout_pad, pk), dtype=w.dtype)
    for tap in range(k_h * k_w):
        ky, kx = divmod(tap, k_w)
        for cb in range(n_cblk):
            c0, c1 = cb * pk, min(c_in, cb * pk + pk)
            out[tap, cb, :, :c_out, :c1 - c0] = w[:, :, c0:c1, ky, kx]
    return out.reshape(-1)


CASES = [  # (Cout, Cin, k, dtype)
    (64, 64, 3, torch.bfloat16),
    (256, 256, 3, torch.bfloat16),
    (64, 64, 1, torch.bfloat16),
    (64, 32, 1, torch.bfloat16),
    (36, 8, 3, torch.bfloat16),     # half a channel block, output padding
    (16, 24, 3, torch.bfloat16),    # 1.5 blocks
    (64, 16, 5, torch.bfloat16),    # 25 taps: the element kernel
    (32, 12, 3, torch.bfloat16),    # Cin not a multiple of 8: the element kernel
    (16, 16, 3, torch.float32),
]


@pytest.mark.parametrize("case", CASES, ids=str)
def test_pack_matches_layout(case):
    c_out, c_in, k, dt = case
    say(f"pack {case}")
    g = torch.Generator().manual_seed(c_out * 1000 + c_in + k)
    ws = [torch.randn(c_out, c_in, k, k, generator=g).to(dt) for _ in range(4)]
    dev = torch.device("cuda:0")
    packed = quan.quan_qconv2d_pack_weights(*[w.to(dev) for w in ws])
    torch.cuda.synchronize()
    got = packed.cpu().view(torch.int16 if dt == torch.bfloat16 else torch.int32).numpy()
    ref = reference_pack(ws, dt)
    assert got.shape == ref.shape
    assert np.array_equal(got, ref), f"pack {case}: {int((got != ref).sum())} of {ref.size} elements differ"


def test_pack_misaligned_sources():
    """Kernels that start 2 bytes past a 16-byte boundary take the element
    kernel and pack the same."""
    c_out, c_in, k = 64, 64, 3
    say("pack misaligned sources")
    g = torch.Generator().manual_seed(7)
    dev = torch.device("cuda:0")
    n = c_out * c_in * k * k
    bufs = [torch.randn(n + 1, generator=g).to(torch.bfloat16).to(dev) for _ in range(4)]
    ws = [b[1:].view(c_out, c_in, k, k) for b in bufs]
    assert all(w.data_ptr() % 16 == 2 for w in ws)
    packed = quan.quan_qconv2d_pack_weights(*ws)
    torch.cuda.synchronize()
    got = packed.cpu().view(torch.int16).numpy()
    assert np.array_equal(got, reference_pack(ws, torch.bfloat16))
