"""Pins of the oracle's direct conv / FC, zero skipping and work counts
against torch/numpy float64 routines, closed forms and hand examples."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth


def _f64(t):
    return t.to(torch.float64)


def _torch_conv(x, w, n, cin, h, wd, cout, kh, kw, sh, sw, ph, pw, dh, dw, groups, bias=None,
                residual=None, act=oracle.ACT_NONE):
    xt = _f64(x).permute(0, 3, 1, 2)                 # NHWC -> NCHW
    wt = _f64(w).permute(0, 3, 1, 2)                 # [co][kh][kw][ci] -> [co][ci][kh][kw]
    y = F.conv2d(xt, wt, None if bias is None else _f64(bias), stride=(sh, sw),
                 padding=(ph, pw), dilation=(dh, dw), groups=groups).permute(0, 2, 3, 1)
    if residual is not None:
        y = y + _f64(residual)
    if act == oracle.ACT_RELU:
        y = torch.relu(y)
    elif act == oracle.ACT_RELU6:
        y = torch.clamp(y, 0, 6)
    return y.numpy()


CONV_CASES = [
    # n, cin, h, w, cout, kh, kw, sh, sw, ph, pw, dh, dw, groups
    (1, 8, 9, 9, 8, 3, 3, 1, 1, 1, 1, 1, 1, 1),
    (2, 4, 7, 10, 6, 3, 3, 2, 2, 1, 1, 1, 1, 1),
    (1, 6, 8, 8, 4, 2, 3, 1, 2, 0, 1, 2, 1, 2),
    (2, 8, 6, 6, 8, 3, 3, 1, 1, 1, 1, 1, 1, 8),      # depthwise
    (1, 8, 9, 9, 8, 3, 3, 2, 2, 1, 1, 1, 1, 8),      # depthwise stride 2
    (1, 3, 15, 15, 5, 7, 7, 2, 2, 3, 3, 1, 1, 1),    # stem-like
    (3, 16, 4, 4, 8, 1, 1, 1, 1, 0, 0, 1, 1, 1),     # pointwise
]


@pytest.mark.parametrize("case", CONV_CASES)
@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("act", [oracle.ACT_NONE, oracle.ACT_RELU, oracle.ACT_RELU6])
def test_conv_vs_torch_float64(case, dt, act):
    n, cin, h, w, cout, kh, kw, sh, sw, ph, pw, dh, dw, groups = case
    seed = CONV_CASES.index(case) * 100 + ["f32", "bf16", "f16"].index(dt) * 10 + act
    x = synth.normal((n, h, w, cin), dt, seed)
    wt = synth.normal((cout, kh, kw, cin // groups), dt, seed + 1)
    bias = synth.normal((cout,), dt, seed + 2)
    ho, wo = oracle.out_dim(h, kh, sh, ph, dh), oracle.out_dim(w, kw, sw, pw, dw)
    res = synth.normal((n, ho, wo, cout), dt, seed + 3)
    y, a, _ = oracle.conv2d(x, wt, n, cin, h, w, cout, kh, kw, sh, sw, ph, pw, dh, dw, groups,
                            bias=bias, residual=res, act=act)
    ref = _torch_conv(x, wt, n, cin, h, w, cout, kh, kw, sh, sw, ph, pw, dh, dw, groups, bias,
                      res, act)
    assert np.all(np.abs(y - ref) <= 1e-13 * a + 1e-300)


def test_conv_delta_input_gives_flipped_kernel():
    # A single 1 at (4, 4) of a 9 x 9 single-channel image: the correlation
    # output around it is the kernel rotated by 180 degrees.
    x = torch.zeros(1, 9, 9, 1)
    x[0, 4, 4, 0] = 1.0
    k = torch.arange(1, 10, dtype=torch.float32).reshape(1, 3, 3, 1)
    y, _, _ = oracle.conv2d(x, k, 1, 1, 9, 9, 1, 3, 3, ph=1, pw=1)
    patch = y[0, 3:6, 3:6, 0]
    assert np.array_equal(patch, np.array([[9, 8, 7], [6, 5, 4], [3, 2, 1]], dtype=np.float64))
    y[0, 3:6, 3:6, 0] = 0
    assert not y.any()


def test_conv_all_ones_interior_and_edges():
    cin = 5
    x = torch.ones(1, 6, 7, cin)
    w = torch.ones(2, 3, 3, cin)
    y, _, _ = oracle.conv2d(x, w, 1, cin, 6, 7, 2, 3, 3, ph=1, pw=1)
    assert np.all(y[0, 1:-1, 1:-1, :] == cin * 9)       # interior: every tap in bounds
    assert np.all(y[0, 0, 1:-1, :] == cin * 6)           # top edge: 2 of 3 rows
    assert np.all(y[0, 0, 0, :] == cin * 4)              # corner: 2 x 2 taps


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
def test_fc_vs_numpy_matmul(dt):
    m, k, n = 5, 67, 9
    x = synth.normal((m, k), dt, 21)
    w = synth.normal((n, k), dt, 22)
    b = synth.normal((n,), dt, 23)
    r = synth.normal((m, n), dt, 24)
    y, a = oracle.fc(x, w, m, k, n, bias=b, residual=r, act=oracle.ACT_RELU)
    ref = np.maximum(_f64(x).numpy() @ _f64(w).numpy().T + _f64(b).numpy() + _f64(r).numpy(), 0)
    assert np.all(np.abs(y - ref) <= 1e-13 * a)


def test_1x1_conv_equals_fc():
    n, h, w, cin, cout = 2, 3, 5, 12, 7
    x = synth.normal((n, h, w, cin), "bf16", 31)
    wt = synth.normal((cout, 1, 1, cin), "bf16", 32)
    yc, ac, _ = oracle.conv2d(x, wt, n, cin, h, w, cout, 1, 1)
    yf, af = oracle.fc(x.reshape(n * h * w, cin), wt.reshape(cout, cin), n * h * w, cin, cout)
    assert np.array_equal(yc.reshape(-1, cout), yf)
    assert np.array_equal(ac.reshape(-1, cout), af)


@pytest.mark.parametrize("rho", [0.0, 0.5, 0.9, 1.0])
@pytest.mark.parametrize("blk", [(1, 1), (1, 4), (2, 8), (1, 16)])
def test_conv_zero_skip_equals_dense_bitwise(rho, blk):
    n, h, w, cin, cout = 2, 6, 6, 16, 4
    x = synth.sparse_nhwc(n, h, w, cin, rho, "bf16", 41)
    wt = synth.normal((cout, 3, 3, cin), "bf16", 42)
    b = synth.normal((cout,), "bf16", 43)
    yd, ad, _ = oracle.conv2d(x, wt, n, cin, h, w, cout, 3, 3, ph=1, pw=1, bias=b,
                              act=oracle.ACT_RELU)
    st = oracle.measure(x, n * h * w, cin, blk[0], blk[1])
    ys, as_, _ = oracle.conv2d(x, wt, n, cin, h, w, cout, 3, 3, ph=1, pw=1, bias=b,
                               act=oracle.ACT_RELU, skip_mask=st["mask"], skip_rows=blk[0],
                               skip_cols=blk[1])
    assert np.array_equal(yd, ys) and np.array_equal(ad, as_)
    if rho == 1.0:
        # every term skipped: output is act(bias) exactly
        ref = np.maximum(_f64(b).numpy(), 0)
        assert np.array_equal(ys, np.broadcast_to(ref, ys.shape))


@pytest.mark.parametrize("pattern", ["iid", "block"])
@pytest.mark.parametrize("rho", [0.0, 0.5, 0.95, 1.0])
def test_fc_zero_skip_equals_dense_bitwise(pattern, rho):
    m, k, n = 24, 96, 10
    x = synth.sparse_matrix(m, k, rho, pattern, "bf16", 51)
    w = synth.normal((n, k), "bf16", 52)
    yd, _ = oracle.fc(x, w, m, k, n)
    for br, bc in ((m, 1), (16, 16), (8, 32)):
        st = oracle.measure(x, m, k, br, bc)
        ys, _ = oracle.fc(x, w, m, k, n, skip_mask=st["mask"], skip_rows=br, skip_cols=bc)
        assert np.array_equal(yd, ys)


def test_fc_executed_blocks_hand_example():
    x = np.zeros((5, 6), dtype=np.float32)
    x[0, 0] = 1      # tile 0 (rows 0-1), block 0 (cols 0-3)
    x[4, 5] = 2      # tile 2 (row 4), block 1 (cols 4-5)
    x[1, 4] = 3      # tile 0, block 1
    assert oracle.fc_executed_blocks(x, 5, 6, 2, 4) == 3
    assert oracle.fc_executed_blocks(np.zeros((5, 6), np.float32), 5, 6, 2, 4) == 0
    assert oracle.fc_executed_blocks(np.ones((5, 6), np.float32), 5, 6, 2, 4) == 6


def test_conv_executed_blocks_extremes_and_hand_example():
    n, h, w, c = 1, 4, 4, 8
    ones = torch.ones(n, h, w, c)
    # dense input, 3x3 pad 1, tiles of 4 outputs = one output row each.  The
    # tiles of output rows 0 and 3 read only padding at the 3 taps of kernel
    # row 0 (resp. 2): 6 taps x 2 channel blocks = 12 each; rows 1 and 2 use
    # all 9 taps: 18 each.  Total 60.
    assert oracle.conv_executed_blocks(ones, n, c, h, w, 3, 3, 1, 1, 1, 1, 1, 1, 4, 4) == 60
    assert oracle.conv_executed_blocks(torch.zeros(n, h, w, c), n, c, h, w, 3, 3, 1, 1, 1, 1,
                                       1, 1, 4, 4) == 0
    # single nonzero at pixel (0, 0), channel 5 (block 1).  The tile of output
    # row 0 reads it at taps (1,1) [ow=0] and (1,0) [ow=1]; the tile of output
    # row 1 at taps (0,1) and (0,0).  4 executed blocks.
    x = torch.zeros(n, h, w, c)
    x[0, 0, 0, 5] = 1.0
    assert oracle.conv_executed_blocks(x, n, c, h, w, 3, 3, 1, 1, 1, 1, 1, 1, 4, 4) == 4


def test_conv_split_executed_blocks_pins():
    """Split execution (each row tile routed on its own): threshold 0 routes
    every tile to the skip path (= conv_executed_blocks), a threshold above 1
    routes every tile to the dense path (tiles x taps x channel blocks), and a
    hand example fixes the per-tile rule, including tiles that straddle
    samples (whose zero fraction is taken over their whole samples)."""
    x = synth.sparse_matrix(2 * 6 * 7, 16, 0.7, "block", "f32", 31).reshape(2, 6, 7, 16)
    args = (2, 16, 6, 7, 3, 3, 1, 1, 1, 1, 1, 1)
    for tr, bc in ((8, 8), (16, 16), (13, 8)):
        skip_all = oracle.conv_executed_blocks(x, *args, tr, bc)
        assert oracle.conv_split_executed_blocks(x, *args, tr, bc, 0.0) == skip_all
        tiles = -(-2 * 6 * 7 // tr)
        assert oracle.conv_split_executed_blocks(x, *args, tr, bc, 2.0) == tiles * 9 * (16 // bc)
    # 1x1 conv, 3 samples of 5 x 5 pixels, 128 channels, blocks of 64: sample 0
    # all zero; sample 1 zero in channels 0-63 only (zero fraction 0.5);
    # sample 2 all zero.  Tiles of 16 rows: t0 = s0, t1 = s0|s1, t2 = s1,
    # t3 = s1|s2, t4 = s2 (zero fractions 1, 0.75, 0.5, 0.75, 1).  A skipping
    # tile that holds sample-1 rows executes 1 block; a dense tile 2; an
    # all-zero skipping tile 0.
    x = torch.zeros(3, 5, 5, 128)
    x[1, :, :, 64:] = 1.0
    a1 = (3, 128, 5, 5, 1, 1, 1, 1, 0, 0, 1, 1, 16, 64)
    assert oracle.conv_split_executed_blocks(x, *a1, 0.4) == 0 + 1 + 1 + 1 + 0
    assert oracle.conv_split_executed_blocks(x, *a1, 0.5) == 0 + 1 + 1 + 1 + 0
    assert oracle.conv_split_executed_blocks(x, *a1, 0.6) == 0 + 1 + 2 + 1 + 0
    assert oracle.conv_split_executed_blocks(x, *a1, 0.8) == 0 + 2 + 2 + 2 + 0
    assert oracle.conv_split_executed_blocks(x, *a1, 1.01) == 2 * 5


def test_conv_at_matches_full():
    n, h, w, cin, cout = 2, 5, 6, 8, 6
    x = synth.normal((n, h, w, cin), "f16", 61)
    wt = synth.normal((cout, 3, 3, cin), "f16", 62)
    r = synth.normal((n, 3, 3, cout), "f16", 63)
    y, a, _ = oracle.conv2d(x, wt, n, cin, h, w, cout, 3, 3, 2, 2, 1, 1, residual=r,
                            act=oracle.ACT_RELU6)
    idx = np.array([0, 7, 31, y.size - 1], dtype=np.int64)
    ys, as_ = oracle.conv2d_at(x, wt, idx, n, cin, h, w, cout, 3, 3, 2, 2, 1, 1, residual=r,
                               act=oracle.ACT_RELU6)
    assert np.array_equal(ys, y.reshape(-1)[idx]) and np.array_equal(as_, a.reshape(-1)[idx])


def test_maxpool_vs_torch():
    x = synth.normal((2, 9, 10, 3), "bf16", 71)
    y = oracle.maxpool2d(x, 2, 3, 9, 10)
    ref = F.max_pool2d(_f64(x).permute(0, 3, 1, 2), 3, 2, 1).permute(0, 2, 3, 1).numpy()
    assert np.array_equal(y, ref)
