"""Pins of the oracle's intensity closed form (Eq. 2) and routing rule."""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_config1_exact_intensity():
    # 3x3 conv, 64 -> 64 channels, 56 x 56, stride 1, pad 1, fp32, bias.
    # MACs = 56*56*64*64*9 = 115,605,504 (hand product).
    # bytes = 4 * (64*56*56 + 64*64*9 + 64*56*56 + 64) = 4 * 438,336 = 1,753,344.
    r = oracle.conv_intensity(1, 64, 56, 56, 64, 3, 3, 1, 1, 1, 1, 1, 1, 1, oracle.F32, 1)
    assert r["macs"] == 115_605_504
    assert r["flops"] == 231_211_008
    assert r["bytes"] == 1_753_344
    assert r["intensity"] == 231_211_008 / 1_753_344


def test_fc_equals_1x1_conv():
    a = oracle.fc_intensity(64, 4096, 4096, oracle.BF16)
    b = oracle.conv_intensity(64, 4096, 1, 1, 4096, 1, 1, dt=oracle.BF16)
    assert a == b
    # hand values: M*K*N = 64 * 4096^2; bytes = 2*(64*4096 + 4096^2 + 64*4096)
    assert a["macs"] == 64 * 4096 * 4096
    assert a["bytes"] == 2 * (2 * 64 * 4096 + 4096 * 4096)


def test_output_extent_vs_torch():
    g = np.random.default_rng(5)
    for _ in range(50):
        h = int(g.integers(1, 20)); k = int(g.integers(1, 6)); s = int(g.integers(1, 4))
        p = int(g.integers(0, 3)); d = int(g.integers(1, 3))
        expect = oracle.out_dim(h, k, s, p, d)
        if expect <= 0:
            continue
        y = torch.nn.functional.conv2d(torch.zeros(1, 1, h, h), torch.zeros(1, 1, k, k),
                                       stride=s, padding=p, dilation=d)
        assert y.shape[-1] == expect


def test_counted_macs_match_closed_form():
    g = np.random.default_rng(11)
    for case in range(40):
        groups = int(g.choice([1, 2, 4]))
        cin = groups * int(g.integers(1, 4)); cout = groups * int(g.integers(1, 4))
        n = int(g.integers(1, 3)); h = int(g.integers(1, 9)); w = int(g.integers(1, 9))
        kh = int(g.integers(1, 4)); kw = int(g.integers(1, 4))
        sh = int(g.integers(1, 3)); sw = int(g.integers(1, 3))
        ph = int(g.integers(0, 2)); pw = int(g.integers(0, 2))
        dh = int(g.integers(1, 3)); dw = int(g.integers(1, 3))
        if oracle.out_dim(h, kh, sh, ph, dh) <= 0 or oracle.out_dim(w, kw, sw, pw, dw) <= 0:
            continue
        x = synth.normal((n, h, w, cin), "f32", seed=case)
        wt = synth.normal((cout, kh, kw, cin // groups), "f32", seed=case + 100)
        _, _, counted = oracle.conv2d(x, wt, n, cin, h, w, cout, kh, kw, sh, sw, ph, pw, dh, dw,
                                      groups)
        closed = oracle.conv_intensity(n, cin, h, w, cout, kh, kw, sh, sw, ph, pw, dh, dw,
                                       groups, oracle.F32)
        assert counted == closed["macs"]


def _resnet18_macs():
    """Sum of Eq. 2 over ResNet-18 at 224 x 224 (He et al. 2016 layer list)."""
    total = 0
    total += oracle.conv_intensity(1, 3, 224, 224, 64, 7, 7, 2, 2, 3, 3)["macs"]
    hw, cin = 56, 64
    for cout, first_stride in ((64, 1), (128, 2), (256, 2), (512, 2)):
        for blk in range(2):
            s = first_stride if blk == 0 else 1
            total += oracle.conv_intensity(1, cin, hw, hw, cout, 3, 3, s, s, 1, 1)["macs"]
            ho = oracle.out_dim(hw, 3, s, 1, 1)
            total += oracle.conv_intensity(1, cout, ho, ho, cout, 3, 3, 1, 1, 1, 1)["macs"]
            if s != 1 or cin != cout:
                total += oracle.conv_intensity(1, cin, hw, hw, cout, 1, 1, s, s, 0, 0)["macs"]
            hw, cin = ho, cout
    total += oracle.fc_intensity(1, 512, 1000)["macs"]
    return total


def test_resnet18_table2():
    with open(os.path.join(GOLDEN, "table2_resnet18.json")) as f:
        gold = json.load(f)
    macs = _resnet18_macs()
    assert macs == 1_814_073_344
    # the paper prints 1.8 "GFLOPs" (two significant figures): Eq. 2 counts MACs
    assert round(macs / 1e9, 1) == gold["giga"]


@pytest.mark.parametrize("bad", [dict(cin=3, groups=2), dict(h=1, kh=3, ph=0)])
def test_invalid_shapes(bad):
    args = dict(n=1, cin=4, h=8, w=8, cout=4, kh=3, kw=3, sh=1, sw=1, ph=1, pw=1, dh=1, dw=1,
                groups=1)
    args.update(bad)
    with pytest.raises(ValueError):
        oracle.conv_intensity(**args)


def test_intensity_overflow_is_invalid():
    with pytest.raises(ValueError):
        oracle.fc_intensity(2**40, 2**20, 2**10)


# ------------------------------------------------------------------ routing

SKIP, BW = 1, 2


def test_route_ties():
    # rho exactly at the threshold routes to the skip path (>=)
    assert oracle.route(50, 100, 0, 0, 10.0, 0, 0.5, 315.0, oracle.ROUTE_ELEMENT) == SKIP | BW
    assert oracle.route(49, 100, 0, 0, 10.0, 0, 0.5, 315.0, oracle.ROUTE_ELEMENT) == BW
    # intensity exactly at the threshold stays on the compute path (strict <)
    assert oracle.route(0, 100, 0, 0, 315.0, 0, 0.5, 315.0, oracle.ROUTE_ELEMENT) == 0
    assert oracle.route(0, 100, 0, 0, np.nextafter(315.0, 0), 0, 0.5, 315.0,
                        oracle.ROUTE_ELEMENT) == BW


def test_route_block_vs_element_mode():
    # element sparsity 0.9 but no all-zero blocks
    assert oracle.route(90, 100, 0, 10, 500.0, 0, 0.5, 315.0, oracle.ROUTE_BLOCK) == 0
    assert oracle.route(90, 100, 0, 10, 500.0, 0, 0.5, 315.0, oracle.ROUTE_ELEMENT) == SKIP
    assert oracle.route(0, 100, 10, 10, 500.0, 0, 1.0, 315.0, oracle.ROUTE_BLOCK) == SKIP


def test_route_depthwise_always_bandwidth():
    assert oracle.route(0, 100, 0, 4, 1e6, 1, 0.5, 315.0) == BW


def test_route_paper_vectors():
    # Section 4 transition example: conv, rho = 0.2, heavy -> dense compute path
    assert oracle.route(20, 100, 0, 1, 973.0, 0, 0.5, 315.0, oracle.ROUTE_ELEMENT) == 0
    # Section 2.2: sparse (> 0.4) and heavy conv stays on the compute side (no BW bit)
    r = oracle.route(45, 100, 0, 1, 400.0, 0, 0.4, 315.0, oracle.ROUTE_ELEMENT)
    assert not (r & BW)
    # Section 2.2: dense, light (BatchNorm-like) operator -> dense bandwidth path
    assert oracle.route(0, 100, 0, 1, 0.5, 0, 0.4, 315.0, oracle.ROUTE_ELEMENT) == BW
    # Section 1 / Section 4: sparse and light -> skip + bandwidth
    assert oracle.route(90, 100, 9, 10, 1.0, 0, 0.4, 315.0) == SKIP | BW


@pytest.mark.parametrize("args", [
    (0, 100, 0, 0, 10.0, 0, 0.5, 315.0, 0),            # block mode without blocks
    (0, 0, 0, 1, 10.0, 0, 0.5, 315.0, 1),              # element mode, numel 0
    (0, 100, 0, 1, 10.0, 0, float("nan"), 315.0, 0),   # NaN threshold
    (0, 100, 0, 1, 10.0, 0, -0.1, 315.0, 0),           # negative threshold
    (0, 100, 0, 1, 10.0, 0, 0.5, 315.0, 7),            # unknown mode
    (101, 100, 0, 1, 10.0, 0, 0.5, 315.0, 1),          # zeros > numel
])
def test_route_invalid(args):
    assert oracle.route(*args) == -1
