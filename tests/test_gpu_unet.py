"""GPU parity of the SDXL UNet ResNet-block kernels through the C ABI (the convolutional
residual units of the appendix "Exact Block-Level Scores", Eq. app-conv-score): GroupNorm +
SiLU and the implicit-GEMM 3x3 convolution against the oracle's definitions."""
import numpy as np
import pytest

import synth
from oracle import model as om
from oracle.numerics import decode, round_bf16

from helpers import rel_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_29505_amd as P
    P.lib()
    return P


def _bf16(x):
    import torch
    return torch.from_numpy(synth.store(np.asarray(x), "bf16").view(np.int16)).view(torch.bfloat16).cuda()


def _host(t):
    import torch
    if t.dtype == torch.bfloat16:
        return decode(t.view(torch.int16).cpu().numpy().view(np.uint16), "bf16")
    return t.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("B,side,C,groups,in_dtype", [(2, 10, 256, 32, "f32"), (2, 10, 256, 32, "bf16"),
                                                      (8, 32, 1280, 32, "f32"), (8, 32, 1280, 32, "bf16"),
                                                      (3, 7, 128, 8, "f32")])
def test_group_norm_silu(P, B, side, C, groups, in_dtype):
    import torch
    rng = np.random.default_rng(C + side)
    N = side * side
    x = rng.standard_normal((B, N, C)) * 2.0 + 0.3
    w = (1 + 0.1 * rng.standard_normal(C)).astype(np.float32)
    b = (0.1 * rng.standard_normal(C)).astype(np.float32)
    if in_dtype == "bf16":
        xd = _bf16(x)
        x = decode(synth.store(x, "bf16"), "bf16")
    else:
        x = x.astype(np.float32).astype(np.float64)
        xd = torch.from_numpy(x.astype(np.float32)).cuda()
    y = torch.empty((B, N, C), dtype=torch.bfloat16, device="cuda")
    P.op_group_norm_silu(xd, y, groups, torch.from_numpy(w).cuda(), torch.from_numpy(b).cuda())
    torch.cuda.synchronize()
    ref = om.silu(om.group_norm(x, groups, w.astype(np.float64), b.astype(np.float64)))
    got = _host(y)
    # one bf16 rounding of the output (at most one ulp from the fp64 value's rounding) plus the
    # fp32 statistics
    assert np.all(np.abs(got - ref) <= 2.0 ** -7 * np.abs(ref) + 1e-5), np.max(np.abs(got - ref))


def _conv_case(rng, B, side, cin, cout):
    x = rng.standard_normal((B, side * side, cin))
    w = rng.standard_normal((cout, 9 * cin)) / np.sqrt(9 * cin)
    return decode(synth.store(x, "bf16"), "bf16"), decode(synth.store(w, "bf16"), "bf16")


@pytest.mark.parametrize("tile", [0, 2, 4, 5])
@pytest.mark.parametrize("B,side,cin,cout", [(2, 10, 256, 256), (1, 5, 64, 128), (3, 9, 128, 192)])
def test_conv3x3(P, tile, B, side, cin, cout):
    """bf16 output of conv + bias + per-sample bias against the oracle's convolution (fp64 on
    the same bf16 operands, then one bf16 rounding); fp32 residual mode to 1e-5."""
    import torch
    rng = np.random.default_rng(cin * 7 + side + tile)
    x, w = _conv_case(rng, B, side, cin, cout)
    bias = (0.1 * rng.standard_normal(cout)).astype(np.float32)
    rowb = rng.standard_normal((B, cout)).astype(np.float32)
    M = B * side * side
    A, W = _bf16(x.reshape(M, cin)), _bf16(w)
    out = torch.empty((M, cout), dtype=torch.bfloat16, device="cuda")
    P.op_conv3x3(A, W, side, out=out, bias=torch.from_numpy(bias).cuda(), rowbias=torch.from_numpy(rowb).cuda(),
                 tile=tile)
    h0 = rng.standard_normal((M, cout)).astype(np.float32)
    h = torch.from_numpy(h0).cuda()
    P.op_conv3x3(A, W, side, h=h, bias=torch.from_numpy(bias).cuda(), tile=tile)
    torch.cuda.synchronize()
    conv = om.conv3x3(x, w, side).reshape(M, cout)
    ref = round_bf16(conv + bias + np.repeat(rowb, side * side, axis=0))
    got = _host(out)
    # one bf16 rounding each (GPU from fp32, oracle from fp64): at most one bf16 ulp apart
    assert np.all(np.abs(got - ref) <= 2.0 ** -7 * np.abs(ref) + 1e-3), np.max(np.abs(got - ref))
    assert rel_err(_host(h), h0 + conv + bias) <= 1e-5


def test_conv3x3_full_shape_sampled(P):
    """The SDXL UNet stage shape (8 samples of a 32 x 32 grid, 1280 channels), at the tile the
    launcher picks: sampled output rows (corners, edges, interior of several samples)
    computed one by one."""
    import torch
    rng = np.random.default_rng(9)
    B, side, c = 8, 32, 1280
    x, w = _conv_case(rng, B, side, c, c)
    M = B * side * side
    A, W = _bf16(x.reshape(M, c)), _bf16(w)
    h = torch.zeros((M, c), dtype=torch.float32, device="cuda")
    P.op_conv3x3(A, W, side, h=h)
    torch.cuda.synchronize()
    got = _host(h)
    img = x.reshape(B, side, side, c)
    for b, y, xx in [(0, 0, 0), (0, 0, 31), (3, 31, 0), (7, 31, 31), (5, 16, 17), (1, 1, 30), (6, 30, 2)]:
        acc = np.zeros(c)
        for ky in range(3):
            for kx in range(3):
                yy, xs = y + ky - 1, xx + kx - 1
                if 0 <= yy < side and 0 <= xs < side:
                    acc += w[:, (3 * ky + kx) * c:(3 * ky + kx + 1) * c] @ img[b, yy, xs]
        row = (b * side + y) * side + xx
        assert rel_err(got[row], acc) <= 1e-5, (b, y, xx)
