"""Layer-level GPU parity: each implicit-GEMM contraction (forward, data
gradient, weight gradient) of hs_layer_gemm against the oracle's convolution
definition, over the shapes the networks use plus ragged edge cases."""
import numpy as np
import pytest
import torch

from oracle import layers as L
from tests.gpu_util import require_gpu, normwise, rne_bf16_bits, bf16_bits_to_f32, log

pytestmark = pytest.mark.gpu

# (n, H, W, C, K, R, stride, pad)
SHAPES = [
    (2, 32, 32, 3, 64, 3, 1, 1),      # stem (C = 3)
    (2, 32, 32, 64, 64, 3, 1, 1),
    (3, 32, 32, 32, 64, 3, 1, 1),     # K slice spans two taps (bf16)
    (2, 16, 16, 64, 128, 3, 2, 1),    # strided 3x3
    (2, 16, 16, 64, 128, 1, 2, 0),    # 1x1 projection
    (5, 4, 4, 512, 512, 3, 1, 1),
    (3, 2, 2, 512, 512, 3, 1, 1),
    (9, 1, 1, 256, 10, 1, 1, 0),      # linear 256 -> 10
    (9, 1, 1, 784, 256, 1, 1, 0),     # linear 784 -> 256
    (7, 1, 1, 512, 512, 1, 1, 0),
    (1, 8, 8, 128, 64, 3, 1, 1),
    (2, 32, 32, 8, 64, 3, 1, 1),      # channel-padded first layer (bf16 slice spans 8 taps)
    (3, 32, 32, 4, 32, 3, 1, 1),      # channel-padded first layer (fp32)
    (2, 8, 8, 512, 256, 1, 2, 0),     # 1x1 strided, wide
    (3, 6, 6, 64, 128, 3, 2, 1),      # strided 3x3 on an even map with ragged tiles
    (3, 8, 8, 128, 128, 3, 1, 1),     # 128-channel 3x3 (32x32 MFMA tiles in the step)
    (2, 16, 16, 128, 128, 3, 1, 1),
    (3, 16, 16, 64, 128, 3, 1, 1),
    (5, 4, 4, 256, 512, 3, 1, 1),
    (7, 1, 1, 512, 256, 1, 1, 0),     # linear with 128+ inputs
    # ResNet-50 bottleneck layers: 1x1 to and from the inner width, the
    # strided 3x3 at the inner width, strided 1x1 projections
    (3, 32, 32, 64, 64, 1, 1, 0),
    (2, 32, 32, 256, 64, 1, 1, 0),
    (2, 32, 32, 64, 256, 1, 1, 0),
    (3, 32, 32, 128, 128, 3, 2, 1),
    (2, 32, 32, 256, 512, 1, 2, 0),
    (3, 16, 16, 512, 128, 1, 1, 0),   # 1.5 tiles of 512 rows
    (5, 8, 8, 1024, 256, 1, 1, 0),    # under one tile
    (3, 4, 4, 512, 2048, 1, 1, 0),
    (7, 4, 4, 2048, 512, 1, 1, 0),
    (5, 8, 8, 512, 512, 3, 2, 1),
    (3, 8, 8, 1024, 2048, 1, 2, 0),
]


def rounded(x, dtype):
    if dtype == "fp32":
        return x.astype(np.float32), torch.from_numpy(x.astype(np.float32)).cuda()
    bits = rne_bf16_bits(x)
    return bf16_bits_to_f32(bits), torch.from_numpy(bits.view(np.int16)).cuda()


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
@pytest.mark.parametrize("mode", [0, 1, 2])
def test_layer_gemm(mode, shape, dtype):
    check_layer_gemm(mode, shape, dtype, packed=False)


# 3x3 stride-1 layers whose 512-row tiles hold whole images (the LDS-patch
# form of the 32x32 MFMA kernel): several tiles with a ragged last one, 64-
# and 128-column tiles, images of 16x16 down to 2x2
PATCH_SHAPES = [
    (9, 16, 16, 128, 128, 3, 1, 1),   # 4.5 tiles of 2 images
    (37, 8, 8, 128, 256, 3, 1, 1),    # 4.6 tiles of 8 images
    (70, 4, 4, 256, 128, 3, 1, 1),    # 2.2 tiles of 32 images
    (130, 2, 2, 512, 512, 3, 1, 1),   # 128 images per tile, 2 left over
    (4, 8, 8, 192, 192, 3, 1, 1),     # 64-column tiles, one partial tile
    (5, 8, 8, 128, 64, 3, 1, 1),
    # stride 2 with bf16 outputs (the data gradient by output parity class)
    (3, 32, 32, 64, 128, 3, 2, 1),
    (9, 16, 16, 128, 256, 3, 2, 1),
    (37, 8, 8, 256, 128, 3, 2, 1),
    (4, 16, 16, 64, 64, 3, 2, 1),
]


# bf16 weight gradients of 3x3 stride-2 layers (the parity-plane patch
# kernel for 16-, 8- and 4-wide outputs): several slices per image, whole-
# image slices, and slices of four images with a ragged last one
WGRAD_S2_SHAPES = [
    (9, 32, 32, 64, 128, 3, 2, 1),
    (4, 32, 32, 128, 64, 3, 2, 1),
    (13, 16, 16, 128, 256, 3, 2, 1),
    (7, 8, 8, 256, 128, 3, 2, 1),
    (18, 8, 8, 64, 64, 3, 2, 1),
]


@pytest.mark.parametrize("shape", WGRAD_S2_SHAPES, ids=[str(s) for s in WGRAD_S2_SHAPES])
def test_layer_wgrad_stride2(shape):
    check_layer_gemm(2, shape, "bf16", packed=False)


# bf16 forward (bf16 output) and data gradient given a scratch buffer: the
# 32x32 MFMA kernel on packed weights wherever the shape allows it
@pytest.mark.parametrize("shape", SHAPES + PATCH_SHAPES, ids=[str(s) for s in SHAPES + PATCH_SHAPES])
@pytest.mark.parametrize("mode", [0, 1])
def test_layer_gemm_packed(mode, shape):
    check_layer_gemm(mode, shape, "bf16", packed=True)


def check_layer_gemm(mode, shape, dtype, packed):
    hs = require_gpu()
    n, H, W, C, K, R, st, pad = shape
    log("layer_gemm mode=%d shape=%s %s%s" % (mode, shape, dtype, " packed" if packed else ""))
    Ho, Wo = (H + 2 * pad - R) // st + 1, (W + 2 * pad - R) // st + 1
    rng = np.random.default_rng(sum(shape) + mode)
    x, xd = rounded(rng.standard_normal((n, H, W, C)), dtype)
    w, wd = rounded(rng.standard_normal((K, R, R, C)) / np.sqrt(R * R * C), dtype)
    dy, dyd = rounded(rng.standard_normal((n, Ho, Wo, K)), dtype)
    x64, w64, dy64 = x.astype(np.float64), w.astype(np.float64), dy.astype(np.float64)
    scratch = torch.empty(1 << 22, device="cuda")
    sp, sf = (scratch.data_ptr(), scratch.numel()) if packed else (0, 0)
    if mode == 0:
        bias = rng.standard_normal(K).astype(np.float32)
        out = torch.empty(n * Ho * Wo * K, device="cuda",
                          dtype=torch.int16 if packed else torch.float32)
        hs.layer_gemm(0, dtype, n, H, W, C, K, R, st, pad, xd.data_ptr(), wd.data_ptr(),
                      out.data_ptr(), torch.from_numpy(bias).cuda().data_ptr(), relu=True,
                      out_f32=not packed, scratch=sp, scratch_floats=sf)
        ref = np.maximum(L.conv_forward(x64, w64, st, pad, bias.astype(np.float64)), 0.0)
    elif mode == 1:
        out = torch.empty(n * H * W * C, device="cuda", dtype=torch.float32 if dtype == "fp32" else torch.int16)
        hs.layer_gemm(1, dtype, n, H, W, C, K, R, st, pad, dyd.data_ptr(), wd.data_ptr(),
                      out.data_ptr(), scratch=sp, scratch_floats=sf)
        ref = L.conv_backward(x64, w64, dy64, st, pad)[0]
    else:
        out = torch.empty(K * R * R * C, device="cuda")
        hs.layer_gemm(2, dtype, n, H, W, C, K, R, st, pad, dyd.data_ptr(), xd.data_ptr(),
                      out.data_ptr(), scratch=scratch.data_ptr(), scratch_floats=scratch.numel())
        ref = L.conv_backward(x64, w64, dy64, st, pad)[1]
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    if got.dtype == np.int16:
        got = bf16_bits_to_f32(got.view(np.uint16))
    err = normwise(got.reshape(-1), ref.reshape(-1))
    log("  normwise err %.3e" % err)
    # bf16 outputs (data gradient, packed forward) carry the output rounding
    tol = 1e-5 if dtype == "fp32" else (5e-3 if mode == 1 or packed else 1e-5)
    assert err <= tol


def test_mfma_loop_probe():
    """hs_probe_mfma_loop (the attainable-rate probe the benchmark reports)
    runs the MFMAs it counts: each wave's outputs add up to 8 x iters x the
    sum of one 32x32x16 product of its operands, sum_k colsum(A)[k] rowsum(B)[k],
    with lane l feeding k block l // 32, elements i = 0..7."""
    hs = require_gpu()
    blocks, iters = 3, 5
    out = torch.zeros(blocks * 512, device="cuda")
    hs.probe_mfma_loop(blocks, iters, out.data_ptr())
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64).reshape(blocks, 8, 64).sum(axis=2)
    for w in range(8):
        t = 64 * w + np.arange(64)
        total = 0.0
        for h in range(2):
            lanes = t[32 * h:32 * h + 32]
            for i in range(8):
                total += float(((lanes + i) % 8).sum()) * float(((3 * lanes + i) % 8).sum())
        np.testing.assert_array_equal(got[:, w], 8 * iters * total)


@pytest.mark.parametrize("nbytes", [16, 4096 + 48, (1 << 24) + 16 * 12345])
def test_copy_probe(nbytes):
    """hs_probe_copy (the attainable-bandwidth probe) copies every byte, with
    a ragged tail past its unrolled loop."""
    hs = require_gpu()
    n = nbytes // 4
    src = torch.arange(n, device="cuda", dtype=torch.int32)
    dst = torch.full((n + 4,), -1, device="cuda", dtype=torch.int32)
    hs.probe_copy(src.data_ptr(), dst.data_ptr(), nbytes)
    torch.cuda.synchronize()
    assert torch.equal(dst[:n], src) and torch.all(dst[n:] == -1)
