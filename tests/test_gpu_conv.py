"""GPU parity of the conv paths (implicit-GEMM MFMA dense / zero-skip,
depthwise bandwidth kernel) and the max-pool glue against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests._util import RTOL, SUBNORMAL_STEP, assert_close

pytestmark = pytest.mark.gpu

DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def _abi():
    from paper_2511_19457_amd import abi
    return abi


def run_conv(x, w, shape, path, bias=None, residual=None, act=0):
    """x NHWC, w [co][kh][kw][ci/g] (CPU tensors).  Returns (y, executed, counts)."""
    abi = _abi()
    dev = torch.device("cuda")
    n, cin, h, wd, cout, kh, kw, sh, sw, ph, pw, dh, dw, groups = shape
    d = abi.conv_desc(n, cin, h, wd, cout, kh, kw, sh, sw, ph, pw, dh, dw, groups, x.dtype,
                      has_bias=bias is not None)
    ho = (h + 2 * ph - dh * (kh - 1) - 1) // sh + 1
    wo = (wd + 2 * pw - dw * (kw - 1) - 1) // sw + 1
    xd = x.to(dev)
    br, bc = abi.sparoa_conv2d_skip_block(d, path)
    counts = torch.zeros(4, dtype=torch.int64, device=dev)
    mask = torch.zeros(abi.sparoa_mask_words(n * h * wd, cin, br, bc), dtype=torch.int32,
                       device=dev)
    c = abi.sparoa_measure_sparsity_sync(xd, n * h * wd, cin, br, bc, 0, counts, mask)
    ws = torch.empty(max(16, abi.sparoa_conv2d_workspace_size(d, path)), dtype=torch.uint8,
                     device=dev)
    y = torch.full((n, ho, wo, cout), float("nan"), dtype=x.dtype, device=dev)
    ex = torch.full((1,), -1, dtype=torch.int64, device=dev)
    abi.sparoa_conv2d(d, path, xd, w.to(dev), None if bias is None else bias.to(dev),
                      None if residual is None else residual.to(dev), act,
                      mask if path & 1 else None, y, ws, ex if path & 1 else None)
    torch.cuda.synchronize()
    return y.cpu(), int(ex.item()), c


def oracle_conv(x, w, shape, bias=None, residual=None, act=0):
    n, cin, h, wd, cout, kh, kw, sh, sw, ph, pw, dh, dw, groups = shape
    y, a, _ = oracle.conv2d(x, w, n, cin, h, wd, cout, kh, kw, sh, sw, ph, pw, dh, dw, groups,
                            bias=bias, residual=residual, act=act)
    return y, a


GEMM_SHAPES = [
    # n, cin, h, w, cout, kh, kw, sh, sw, ph, pw, dh, dw, groups
    (1, 64, 14, 14, 64, 3, 3, 1, 1, 1, 1, 1, 1, 1),
    (2, 32, 9, 11, 48, 3, 3, 2, 2, 1, 1, 1, 1, 1),
    (1, 128, 7, 7, 200, 1, 1, 1, 1, 0, 0, 1, 1, 1),
    (3, 24, 10, 10, 144, 1, 1, 1, 1, 0, 0, 1, 1, 1),   # MobileNetV2-like pointwise
    (1, 3, 23, 23, 16, 7, 7, 2, 2, 3, 3, 1, 1, 1),     # stem: c_in % 8 != 0
    (1, 16, 12, 12, 32, 3, 3, 1, 1, 2, 2, 2, 2, 1),    # dilation 2
    (2, 256, 8, 8, 64, 1, 1, 2, 2, 0, 0, 1, 1, 1),     # strided projection
]


@pytest.mark.parametrize("dt", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("shape", GEMM_SHAPES)
def test_conv_dense_vs_oracle(dt, shape):
    seed = GEMM_SHAPES.index(shape) * 10 + list(DT).index(dt)
    n, cin, h, wd, cout, kh, kw, sh, sw, ph, pw, dh, dw, g = shape
    ho = (h + 2 * ph - dh * (kh - 1) - 1) // sh + 1
    wo = (wd + 2 * pw - dw * (kw - 1) - 1) // sw + 1
    x = synth.relu_normal((n, h, wd, cin), dt, seed)
    w = synth.he_normal((cout, kh, kw, cin), kh * kw * cin, dt, seed + 1)
    b = synth.normal((cout,), dt, seed + 2)
    r = synth.normal((n, ho, wo, cout), dt, seed + 3)
    y, _, _ = run_conv(x, w, shape, 0, bias=b, residual=r, act=1)
    yr, ar = oracle_conv(x, w, shape, bias=b, residual=r, act=1)
    assert_close(y, yr, ar, RTOL[DT[dt]], f"conv {shape} {dt}")


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("rho", [0.0, 0.9, 0.999, 1.0])
@pytest.mark.parametrize("shape", [GEMM_SHAPES[0], GEMM_SHAPES[2], GEMM_SHAPES[6],
                                   (2, 64, 16, 16, 128, 3, 3, 1, 1, 1, 1, 1, 1, 1),
                                   GEMM_SHAPES[3], GEMM_SHAPES[4], GEMM_SHAPES[5]])
def test_conv_skip_equals_dense_and_oracle(dt, rho, shape):
    n, cin, h, wd, cout, kh, kw, sh, sw, ph, pw, dh, dw, g = shape
    x = synth.sparse_nhwc(n, h, wd, cin, rho, dt, int(rho * 1000) + cin)
    w = synth.he_normal((cout, kh, kw, cin), kh * kw * cin, dt, cout)
    yd, _, _ = run_conv(x, w, shape, 0, act=1)
    ys, ex, _ = run_conv(x, w, shape, 1, act=1)
    assert torch.equal(yd, ys)
    yr, ar = oracle_conv(x, w, shape, act=1)
    assert_close(ys, yr, ar, RTOL[DT[dt]], f"skip conv {shape}")
    abi = _abi()
    d = abi.conv_desc(n, cin, h, wd, cout, kh, kw, sh, sw, ph, pw, dh, dw, g, DT[dt])
    tr, kc = abi.sparoa_conv2d_tiling(d, 1)
    if cin % kc == 0:
        assert ex == oracle.conv_executed_blocks(x, n, cin, h, wd, kh, kw, sh, sw, ph, pw, dh,
                                                 dw, tr, kc)
    if rho == 1.0:
        assert ex == 0


DW_SHAPES = [
    (2, 32, 12, 12, 32, 3, 3, 1, 1, 1, 1, 1, 1, 32),
    (1, 96, 15, 15, 96, 3, 3, 2, 2, 1, 1, 1, 1, 96),
    (1, 144, 8, 9, 144, 3, 3, 1, 1, 1, 1, 1, 1, 144),  # even Ho, odd Wo: 2 x 1 items
    (2, 48, 6, 10, 48, 3, 3, 1, 1, 1, 1, 1, 1, 48),    # even Ho, Wo 10: 2 x 2 items
    (1, 12, 7, 7, 12, 5, 5, 1, 1, 2, 2, 1, 1, 12),     # runtime-window kernel
    (1, 5, 6, 6, 5, 3, 3, 1, 1, 1, 1, 1, 1, 5),        # channels % 8 != 0
    (3, 24, 14, 13, 24, 3, 3, 2, 2, 1, 1, 1, 1, 24),   # stride 2, ragged pixel runs
    (2, 16, 5, 3, 16, 3, 3, 1, 1, 1, 1, 1, 1, 16),     # row narrower than a run
    (1, 40, 9, 9, 40, 3, 3, 1, 1, 1, 1, 2, 2, 40),     # dilation 2: general kernel
    (2, 32, 37, 21, 32, 3, 3, 1, 1, 1, 1, 1, 1, 32),   # stride 1: ragged row and column tiles
    (1, 88, 13, 11, 88, 3, 3, 1, 1, 1, 1, 1, 1, 88),   # 11 vectors per pixel: 1-vector tiles
]


@pytest.mark.parametrize("dt", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("shape", DW_SHAPES)
def test_depthwise_vs_oracle(dt, shape):
    n, cin, h, wd, cout, kh, kw, sh, sw, ph, pw, dh, dw, g = shape
    ho = (h + 2 * ph - dh * (kh - 1) - 1) // sh + 1
    wo = (wd + 2 * pw - dw * (kw - 1) - 1) // sw + 1
    seed = DW_SHAPES.index(shape) * 7
    x = synth.relu_normal((n, h, wd, cin), dt, seed)
    w = synth.he_normal((cout, kh, kw, 1), kh * kw, dt, seed + 1)
    b = synth.normal((cout,), dt, seed + 2)
    r = synth.normal((n, ho, wo, cout), dt, seed + 3)
    for path in (2, 3):
        y, _, _ = run_conv(x, w, shape, path, bias=b, residual=r, act=2)
        yr, ar = oracle_conv(x, w, shape, bias=b, residual=r, act=2)
        assert_close(y, yr, ar, RTOL[DT[dt]], f"depthwise {shape} {dt}")


@pytest.mark.parametrize("stride", [1, 2])
def test_depthwise_grid_stride_loop(stride):
    """More lane items than the grid holds (over 2^20): lanes loop over items;
    the first and last images are checked against the oracle."""
    n, c, hw = 160 * stride, 16, 128
    shape = (n, c, hw, hw, c, 3, 3, stride, stride, 1, 1, 1, 1, c)
    x = synth.relu_normal((n, hw, hw, c), "bf16", 91 + stride)
    w = synth.he_normal((c, 3, 3, 1), 9, "bf16", 93)
    y, _, _ = run_conv(x, w, shape, 2, act=1)
    for sel in (slice(0, 2), slice(n - 2, n)):
        sub = (2,) + shape[1:]
        yr, ar = oracle_conv(x[sel].contiguous(), w, sub, act=1)
        assert_close(y[sel], yr, ar, RTOL[torch.bfloat16], f"depthwise loop s{stride} {sel}")


# Inputs of at most 4 channels (image stems) run the direct small-channel kernel.
SMALL_C_SHAPES = [
    (2, 3, 64, 64, 64, 7, 7, 2, 2, 3, 3, 1, 1, 1),     # ResNet stem, Wo 32
    (2, 3, 50, 50, 32, 3, 3, 2, 2, 1, 1, 1, 1, 1),     # MobileNetV2 stem, ragged row block
    (1, 1, 20, 37, 16, 4, 4, 1, 1, 1, 2, 1, 1, 1),     # one channel, even kw, stride 1
    (1, 4, 9, 256, 64, 5, 5, 2, 2, 2, 2, 1, 1, 1),     # four channels, Wo 128 (8 row blocks)
]


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("shape", SMALL_C_SHAPES)
def test_small_c_conv_vs_oracle_and_skip(dt, shape):
    """Dense output against the oracle (bias, residual, ReLU); the skip path
    equal to the dense path bit for bit on an input whose top half is zero
    (some k-steps skipped), and executing nothing on an all-zero input."""
    abi = _abi()
    n, cin, h, wd, cout, kh, kw, sh, sw, ph, pw, dh, dw, g = shape
    d = abi.conv_desc(*shape, DT[dt])
    assert abi.sparoa_conv2d_tiling(d, 1) == (16, 32)
    ho = (h + 2 * ph - kh) // sh + 1
    wo = (wd + 2 * pw - kw) // sw + 1
    seed = 1500 + SMALL_C_SHAPES.index(shape)
    x = synth.relu_normal((n, h, wd, cin), dt, seed)
    x[:, : h // 2] = 0
    w = synth.he_normal((cout, kh, kw, cin), kh * kw * cin, dt, seed + 1)
    b = synth.normal((cout,), dt, seed + 2)
    r = synth.normal((n, ho, wo, cout), dt, seed + 3)
    yd, _, _ = run_conv(x, w, shape, 0, bias=b, residual=r, act=1)
    ys, ex, _ = run_conv(x, w, shape, 1, bias=b, residual=r, act=1)
    assert torch.equal(yd, ys)
    total = n * ho * -(-wo // 16) * -(-(kh * -(-kw // 2)) // 4)   # (row block, k-step) pairs
    assert 0 < ex < total
    yr, ar = oracle_conv(x, w, shape, bias=b, residual=r, act=1)
    assert_close(yd, yr, ar, RTOL[DT[dt]], f"small-c conv {shape} {dt}")
    z = torch.zeros_like(x)
    yz, exz, _ = run_conv(z, w, shape, 1, bias=b, act=1)
    yzd, _, _ = run_conv(z, w, shape, 0, bias=b, act=1)
    assert exz == 0 and torch.equal(yz, yzd)


def test_resnet50_stem_full_size():
    """The ResNet-50 stem at batch 32 (224 x 224 x 3 -> 112 x 112 x 64, 7x7/2),
    bf16: sampled outputs against the oracle, skip path equal to dense."""
    shape = (32, 3, 224, 224, 64, 7, 7, 2, 2, 3, 3, 1, 1, 1)
    x = synth.normal((32, 224, 224, 3), "bf16", synth.seed_for(3, 1))
    w = synth.he_normal((64, 7, 7, 3), 147, "bf16", synth.seed_for(3, 2))
    yd, _, _ = run_conv(x, w, shape, 0, act=1)
    ys, _, _ = run_conv(x, w, shape, 1, act=1)
    assert torch.equal(yd, ys)
    total = yd.numel()
    rng = np.random.default_rng(77)
    idx = np.unique(np.concatenate([rng.integers(0, total, size=4096), [0, total - 1]]))
    yr, ar = oracle.conv2d_at(x, w, idx, *shape, act=1)
    yg = yd.reshape(-1)[idx].float().numpy().astype(np.float64)
    bound = RTOL[torch.bfloat16] * ar + SUBNORMAL_STEP[torch.bfloat16]
    assert np.all(np.abs(yg - yr) <= bound), float(np.max(np.abs(yg - yr) - bound))


def test_config1_full():
    """Single 3x3 conv 64 -> 64 at 56 x 56, fp32, ReLU(N(0,1)) input."""
    shape = (1, 64, 56, 56, 64, 3, 3, 1, 1, 1, 1, 1, 1, 1)
    x = synth.relu_normal((1, 56, 56, 64), "f32", synth.seed_for(1, 0))
    w = synth.he_normal((64, 3, 3, 64), 576, "f32", synth.seed_for(1, 1))
    b = torch.zeros(64)
    y, _, c = run_conv(x, w, shape, 0, bias=b)
    yr, ar = oracle_conv(x, w, shape, bias=b)
    assert_close(y, yr, ar, 1e-5, "config 1")
    ref = oracle.measure(x, 3136, 64)
    assert c["zeros"] == ref["zeros"]


@pytest.mark.parametrize("dt", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("shape", [(2, 17, 18, 64), (3, 29, 23, 24), (2, 9, 7, 12), (1, 4, 4, 8)],
                         ids=["c64", "c24-odd-hw", "c12-general", "tiny"])
def test_maxpool_vs_oracle(dt, shape):
    # whole 16-byte channel vectors: the 32-bit multiply-shift kernel; C = 12
    # in a 16-bit type: the general one
    abi = _abi()
    n, h, w, c = shape
    x = synth.normal((n, h, w, c), dt, 123 + c)
    ho, wo = (h - 1) // 2 + 1, (w - 1) // 2 + 1
    y = torch.empty(n, ho, wo, c, dtype=DT[dt], device="cuda")
    abi.sparoa_maxpool2d(x.cuda(), n, c, h, w, 3, 2, 1, y)
    torch.cuda.synchronize()
    ref = oracle.maxpool2d(x, n, c, h, w)
    assert np.array_equal(y.float().cpu().numpy().astype(np.float64), ref)


# Shapes that make the tile chooser pick each tile of the 64-channel-chunk
# kernel (expected tile rows in the last field).
IG_SHAPES = [
    ((2, 64, 64, 64, 1024, 1, 1, 1, 1, 0, 0, 1, 1, 1), 128),   # 128 x 256, 1x1, wide N
    ((4, 128, 57, 55, 512, 1, 1, 1, 1, 0, 0, 1, 1, 1), 128),   # 128 x 256, 1x1, ragged M
    ((2, 64, 80, 64, 640, 1, 1, 1, 1, 0, 0, 1, 1, 1), 128),    # 128 x 128, 1x1, N % 256 != 0
    ((6, 64, 61, 67, 256, 3, 3, 1, 1, 1, 1, 1, 1, 1), 128),    # 128 x 128, 3x3, ragged M
    ((1, 64, 64, 64, 1000, 1, 1, 1, 1, 0, 0, 1, 1, 1), 128),   # 128 x 64, ragged N
    ((4, 64, 128, 128, 64, 3, 3, 1, 1, 1, 1, 1, 1, 1), 128),   # 128 x 64, N = 64
    ((2, 64, 127, 129, 64, 3, 3, 1, 1, 1, 1, 1, 1, 1), 128),   # 128 x 64, ragged M
    ((1, 128, 32, 64, 1024, 1, 1, 1, 1, 0, 0, 1, 1, 1), 128),  # 128 x 64, wide N
    ((2, 256, 9, 9, 96, 3, 3, 2, 2, 1, 1, 1, 1, 1), 64),       # 64 x 64, split-K
    ((2, 128, 9, 9, 96, 3, 3, 2, 2, 1, 1, 1, 1, 1), 64),       # 64 x 64, too few chunks to split
    ((1, 192, 7, 7, 36, 3, 3, 1, 1, 1, 1, 1, 1, 1), 64),       # 64 x 64, N % 8 != 0
    # C_in % 64 != 0: a tap's last chunk is partial
    ((2, 96, 14, 14, 576, 1, 1, 1, 1, 0, 0, 1, 1, 1), 64),     # 1x1, 96 = 64 + 32
    ((1, 160, 7, 7, 960, 1, 1, 1, 1, 0, 0, 1, 1, 1), 64),      # 1x1, 160 = 2 x 64 + 32
    ((32, 96, 28, 28, 128, 1, 1, 1, 1, 0, 0, 1, 1, 1), 128),   # 128 x 64, 1x1
    ((2, 56, 19, 21, 72, 3, 3, 1, 1, 1, 1, 1, 1, 1), 64),      # 3x3, 56 < 64: one partial chunk per tap
    ((1, 200, 9, 11, 64, 3, 3, 2, 2, 1, 1, 1, 1, 1), 64),      # 3x3 stride 2, 200 = 3 x 64 + 8, split-K
]


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("case", IG_SHAPES)
def test_chunk64_tiles_vs_oracle_and_skip(dt, case):
    """Every tile of the 64-channel-chunk kernel: sampled outputs against the
    oracle (bias, residual, ReLU), and the skip path equal to the dense path
    bit for bit on an input whose second image and first 64 channels are
    zero (whole chunks skipped)."""
    shape, rows = case
    abi = _abi()
    n, cin, h, wd, cout, kh, kw, sh, sw, ph, pw, dh, dw, g = shape
    d = abi.conv_desc(n, cin, h, wd, cout, kh, kw, sh, sw, ph, pw, dh, dw, g, DT[dt])
    assert abi.sparoa_conv2d_tiling(d, 0) == (rows, 64)
    ho = (h + 2 * ph - dh * (kh - 1) - 1) // sh + 1
    wo = (wd + 2 * pw - dw * (kw - 1) - 1) // sw + 1
    seed = 900 + IG_SHAPES.index(case)
    x = synth.relu_normal((n, h, wd, cin), dt, seed)
    if n > 1:
        x[1:] = 0
    if cin >= 128:
        x[..., :64] = 0
    w = synth.he_normal((cout, kh, kw, cin), kh * kw * cin, dt, seed + 1)
    b = synth.normal((cout,), dt, seed + 2)
    r = synth.normal((n, ho, wo, cout), dt, seed + 3)
    yd, _, _ = run_conv(x, w, shape, 0, bias=b, residual=r, act=1)
    ys, ex, _ = run_conv(x, w, shape, 1, bias=b, residual=r, act=1)
    assert torch.equal(yd, ys)
    total = yd.numel()
    rng = np.random.default_rng(seed)
    idx = np.unique(np.concatenate([rng.integers(0, total, size=3000), [0, total - 1]]))
    yr, ar = oracle.conv2d_at(x, w, idx, n, cin, h, wd, cout, kh, kw, sh, sw, ph, pw, dh, dw, g,
                              bias=b, residual=r, act=1)
    yg = yd.reshape(-1)[idx].float().numpy().astype(np.float64)
    bound = RTOL[DT[dt]] * ar + SUBNORMAL_STEP[DT[dt]]
    assert np.all(np.abs(yg - yr) <= bound), float(np.max(np.abs(yg - yr) - bound))
    full = oracle.conv_executed_blocks(x, n, cin, h, wd, kh, kw, sh, sw, ph, pw, dh, dw, rows, 64)
    assert ex == full
