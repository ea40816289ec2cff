"""The bandwidth-path pointwise (1x1) kernel: every MobileNetV2 pointwise
shape and the ResNet-50 1x1 shapes it serves, against the oracle's direct
conv (element by element within the dtype's tolerance); the skip form equals
the dense form bit for bit and executes exactly the (16-pixel, 32-channel)
blocks the oracle counts; the fused output measurement equals the oracle's
measurement of the output; FCs over many rows on the bandwidth path run it
too."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests._util import RTOL, assert_close

pytestmark = pytest.mark.gpu


def _abi():
    from paper_2511_19457_amd import abi
    return abi


# (c_in, c_out, h, stride, residual) of every MobileNetV2 expand / project
# conv the kernel serves (c_in <= 256 and the weights in at most four 48 KB
# LDS slices), at its own spatial size
MBV2 = [(32, 16, 112, 1, False), (16, 96, 112, 1, False), (96, 24, 56, 1, False),
        (24, 144, 56, 1, False), (144, 24, 56, 1, True), (144, 32, 28, 1, False),
        (32, 192, 28, 1, False), (192, 32, 28, 1, True)]
# 1x1 convs of ResNet-50 widths it serves (bandwidth-routed at the bf16 ridge;
# with 64 output channels or more only from 32768 pixels: below, the implicit
# GEMM serves them)
R50 = [(64, 64, 56, 1, False), (64, 256, 56, 1, True), (128, 32, 56, 1, False)]


def _batch(cin, cout, h, s, small):
    """A batch the pointwise kernel serves: `small` images, or enough for
    32768 output pixels where the implicit GEMM would take fewer."""
    ho = (h - 1) // s + 1
    if cout >= 64 and (cin % 64 == 0 or cin >= 48):
        return max(small, -(-32768 // (ho * ho)))
    return small


def test_shapes_beyond_the_kernel_run_the_implicit_gemm():
    abi = _abi()
    # (weights beyond four LDS slices, K > 256, several slices over few
    # pixels, or fewer than 32768 pixels with 64 output channels or more)
    for cin, cout, h, s in ((160, 960, 7, 1), (256, 512, 56, 2), (384, 64, 14, 1),
                            (96, 576, 14, 1), (64, 384, 14, 1), (128, 512, 28, 1),
                            (192, 64, 14, 1), (256, 64, 56, 1), (64, 256, 56, 1),
                            (64, 64, 56, 1), (128, 128, 28, 1)):
        d = abi.conv_desc(2, cin, h, h, cout, 1, 1, s, s, 0, 0, 1, 1, 1, torch.bfloat16)
        assert abi.sparoa_conv2d_tiling(d, abi.PATH_DENSE_BW) != (16, 32)


def _case(abi, dev, cin, cout, h, s, with_res, dt, n, seed, act):
    tdt = torch.float16 if dt == "f16" else torch.bfloat16
    d = abi.conv_desc(n, cin, h, h, cout, 1, 1, s, s, 0, 0, 1, 1, 1, tdt)
    assert abi.sparoa_conv2d_tiling(d, abi.PATH_DENSE_BW) == (16, 32), "pointwise kernel serves it"
    ho = (h - 1) // s + 1
    x = synth.relu_normal((n, h, h, cin), dt, seed)
    w = synth.he_normal((cout, 1, 1, cin), cin, dt, seed + 1)
    r = synth.normal((n, ho, ho, cout), dt, seed + 2) if with_res else None
    yr, ar, _ = oracle.conv2d(x, w, n, cin, h, h, cout, 1, 1, s, s, act=act, residual=r)
    return d, tdt, ho, x, w, r, yr, ar


@pytest.mark.parametrize("shape", MBV2 + R50)
def test_pointwise_vs_oracle(shape):
    abi = _abi()
    dev = torch.device("cuda")
    cin, cout, h, s, with_res = shape
    dt = "f16" if shape in MBV2 else "bf16"
    n = _batch(cin, cout, h, s, 2 if h >= 56 else 3)
    seed = 2100 + 10 * (MBV2 + R50).index(shape)
    act = abi.ACT_RELU6 if dt == "f16" else abi.ACT_RELU
    d, tdt, ho, x, w, r, yr, ar = _case(abi, dev, cin, cout, h, s, with_res, dt, n, seed, act)
    xd, wd = x.to(dev), w.to(dev)
    rd = r.to(dev) if r is not None else None
    y = torch.full((n, ho, ho, cout), float("nan"), dtype=tdt, device=dev)
    abi.sparoa_conv2d(d, abi.PATH_DENSE_BW, xd, wd, None, rd, act, None, y)
    torch.cuda.synchronize()
    assert_close(y, yr, ar, RTOL[tdt], f"pointwise {shape}")
    # skip form: same bits, executed blocks as the oracle counts them
    counts = torch.zeros(4, dtype=torch.int64, device=dev)
    mask = torch.zeros(abi.sparoa_mask_words(n * h * h, cin, 1, 8), dtype=torch.int32, device=dev)
    abi.sparoa_measure_sparsity(xd, n * h * h, cin, 1, 8, 0, counts, mask)
    y2 = torch.full_like(y, float("nan"))
    ex = torch.full((1,), -1, dtype=torch.int64, device=dev)
    abi.sparoa_conv2d(d, abi.PATH_SKIP_BW, xd, wd, None, rd, act, mask, y2, None, ex)
    torch.cuda.synchronize()
    assert torch.equal(y, y2), f"skip != dense {shape}"
    want = oracle.conv_executed_blocks(x, n, cin, h, h, 1, 1, s, s, 0, 0, 1, 1, 16, 32)
    assert int(ex.item()) == want, shape


def _fresh_counts(rows, cols, dev):
    nb = rows * -(-cols // 8)
    return torch.tensor([0, rows * cols, nb, nb], dtype=torch.int64, device=dev)


@pytest.mark.parametrize("shape,n", [((16, 96, 112, 1, False), 2), ((144, 24, 56, 1, True), 3),
                                     ((24, 144, 56, 1, False), 1), ((32, 384, 112, 1, False), 3),
                                     ((64, 256, 56, 1, True), 2), ((32, 16, 37, 2, False), 3),
                                     ((256, 32, 23, 1, False), 5)])
def test_pointwise_routed_measured(shape, n):
    """Device-routed, output-measuring calls on the pointwise kernel (fused
    measurement for one weight slice, a standalone pass for two (32 -> 384);
    ragged last tiles; stride 2): counts and bitmap equal the oracle's
    measurement of y, y equals the fixed-path call's, the commit words are
    left zero."""
    abi = _abi()
    dev = torch.device("cuda")
    cin, cout, h, s, with_res = shape
    n = _batch(cin, cout, h, s, n)
    seed = 2400 + 10 * cin + cout
    d, tdt, ho, x, w, r, yr, ar = _case(abi, dev, cin, cout, h, s, with_res, "bf16", n, seed,
                                        abi.ACT_RELU)
    xd, wd = x.to(dev), w.to(dev)
    rd = r.to(dev) if r is not None else None
    counts = torch.zeros(4, dtype=torch.int64, device=dev)
    mask = torch.zeros(abi.sparoa_mask_words(n * h * h, cin, 1, 8), dtype=torch.int32, device=dev)
    abi.sparoa_measure_sparsity(xd, n * h * h, cin, 1, 8, 0, counts, mask)
    rows = n * ho * ho
    commit = torch.zeros(abi.COMMIT_WORDS_BYTES // 8, dtype=torch.int64, device=dev)
    for s_thr in (0.0, 2.0):
        y = torch.full((n, ho, ho, cout), float("nan"), dtype=tdt, device=dev)
        y_counts = _fresh_counts(rows, cout, dev)
        y_mask = torch.full((abi.sparoa_mask_words(rows, cout, 1, 8),), -1, dtype=torch.int32,
                            device=dev)
        path = torch.full((1,), -1, dtype=torch.int32, device=dev)
        # intensity threshold far above the layer's: the bandwidth path
        abi.sparoa_conv2d_routed_measured(d, s_thr, 1e9, abi.ROUTE_BLOCK, counts, xd, wd, None,
                                          rd, abi.ACT_RELU, mask, y, y_counts, y_mask, None, path,
                                          commit)
        y2 = torch.full_like(y, float("nan"))
        p = abi.PATH_SKIP_BW if s_thr == 0.0 else abi.PATH_DENSE_BW
        abi.sparoa_conv2d(d, p, xd, wd, None, rd, abi.ACT_RELU, mask, y2)
        torch.cuda.synchronize()
        assert int(path.item()) == p
        assert torch.equal(y, y2)
        assert_close(y, yr, ar, RTOL[tdt], f"{shape} s_thr {s_thr}")
        ref = oracle.measure(y.cpu(), rows, cout, 1, 8)
        assert y_counts.cpu().tolist() == [ref["zeros"], ref["numel"], ref["zero_blocks"],
                                           ref["num_blocks"]], (shape, s_thr)
        assert np.array_equal(y_mask.cpu().numpy().view(np.uint32), ref["mask"]), (shape, s_thr)
        assert int(commit.count_nonzero().item()) == 0


def test_fc_over_many_rows_on_the_bandwidth_path():
    """An FC with many rows (32768 or more: below, the implicit GEMM serves
    it) on the bandwidth path is the 1x1 conv over m pixels and runs the
    pointwise kernel (w in [n][k])."""
    abi = _abi()
    dev = torch.device("cuda")
    m, k, n = 33000, 128, 96
    assert abi.sparoa_fc_tiling(abi.fc_desc(1000, k, n, abi.BF16), abi.PATH_DENSE_BW) != (16, 32)
    d = abi.fc_desc(m, k, n, abi.BF16)
    assert not abi.sparoa_fc_uses_packed(d, abi.PATH_DENSE_BW)
    assert abi.sparoa_fc_tiling(d, abi.PATH_DENSE_BW) == (16, 32)
    x = synth.sparse_matrix(m, k, 0.6, "block", "bf16", 2500)
    w = synth.normal((n, k), "bf16", 2501, std=k ** -0.5)
    b = synth.normal((n,), "bf16", 2502)
    d = abi.fc_desc(m, k, n, abi.BF16, has_bias=1)
    y = torch.full((m, n), float("nan"), dtype=torch.bfloat16, device=dev)
    abi.sparoa_fc(d, abi.PATH_DENSE_BW, x.to(dev), w.to(dev), b.to(dev), None, abi.ACT_NONE, None,
                  y)
    torch.cuda.synchronize()
    yr, ar = oracle.fc(x, w, m, k, n, bias=b)
    assert_close(y, yr, ar, RTOL[torch.bfloat16], "fc on the pointwise kernel")
