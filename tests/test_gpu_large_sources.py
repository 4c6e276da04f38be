"""Matrix products whose A source spans 2 GiB or more.

The GEMM kernels reach their operands through buffer descriptors, whose range
is below 2 GiB: offsets past it read as zeros, which is how convolution
padding taps are formed.  Larger sources therefore run as row chunks of whole
samples.  These cases put chunk boundaries inside the batch and check sampled
outputs (border pixels, whose padding taps must read zeros, the samples on
either side of a boundary, the last sample) against the oracle's float32
layers on the same float16 values.  Inputs are drawn on the device with a
seeded generator."""
import numpy as np
import pytest
import torch

from oracle import unet as U

pytestmark = pytest.mark.gpu


def _randn(shape, seed, scale=1.0):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return (torch.randn(shape, generator=g, device="cuda") * scale).half()


def test_linear_over_2gib_source():
    import paper_2312_04429_amd as P
    M, K, N = 1_700_000, 640, 64  # A = 2.18e9 bytes
    print(f"op linear M={M} N={N} K={K} (A {M * K * 2 / 2**30:.2f} GiB)", flush=True)
    x = _randn((M, K), 1)
    w = _randn((N, K), 2, 0.05)
    b = torch.linspace(-1, 1, N, device="cuda")
    out = P.nv_op_linear(x, w, b)
    torch.cuda.synchronize()
    per = (2**31 - 1) // (K * 2)  # rows per chunk
    rows = sorted({0, 1, per - 1, per, per + 1, M // 2, M - 2, M - 1})
    idx = torch.tensor(rows, device="cuda")
    xs = x[idx].float().cpu().numpy()
    ref = U.linear(xs, w.float().cpu().numpy(), b.cpu().numpy())
    got = out[idx].float().cpu().numpy()
    np.testing.assert_allclose(got, ref, rtol=2e-3, atol=2e-3 * np.abs(ref).max())


@pytest.mark.parametrize("B,H,C1,C2,upsample", [(420, 64, 640, 320, 0), (1650, 32, 640, 0, 1)])
def test_conv3x3_over_2gib_source(B, H, C1, C2, upsample):
    import paper_2312_04429_amd as P
    Cout = 64
    print(f"op conv3x3 B={B} H=W={H} Cin={C1}+{C2} upsample={upsample} "
          f"(src {B * H * H * C1 * 2 / 2**30:.2f} GiB)", flush=True)
    x = _randn((B, H, H, C1), 3)
    x2 = _randn((B, H, H, C2), 4) if C2 else None
    cin = C1 + C2
    w = _randn((Cout, 3, 3, cin), 5, 0.05)
    b = torch.linspace(-1, 1, Cout, device="cuda")
    out = P.nv_op_conv3x3(x, w, b, upsample=bool(upsample), x2=x2)
    torch.cuda.synchronize()
    per = (2**31 - 1) // (H * H * C1 * 2)  # samples per chunk
    wn = w.float().cpu().numpy().transpose(0, 3, 1, 2)  # [Cout][Cin][3][3]
    bn = b.cpu().numpy()
    for s in sorted({0, per - 1, per, B - 1}):
        xs = x[s].float().cpu().numpy()
        if C2:
            xs = np.concatenate([xs, x2[s].float().cpu().numpy()], axis=-1)
        xs = xs.transpose(2, 0, 1)  # [Cin][H][W]
        if upsample:
            xs = U.upsample_nearest2(xs)
        ref = U.conv3x3(xs, wn, bn).transpose(1, 2, 0)  # [Ho][Wo][Cout]
        got = out[s].float().cpu().numpy()
        np.testing.assert_allclose(got, ref, rtol=2e-3, atol=2e-3 * np.abs(ref).max(),
                                   err_msg=f"sample {s}")
