"""Pins of the oracle's tolerance scale A = |bias| + sum |x w| (+ |residual|).

Every element-wise parity bound of the GPU tests is rtol * A, so A must not
come from the oracle alone: here it is recomputed with torch / numpy float64
routines on the absolute values of the same decoded inputs (a convolution of
|x| with |w| is exactly the sum of |x w| over the taps, because every product
of magnitudes is a magnitude of a product), for the full conv, the sampled
conv, the FC, and the zero-skipping forms.  A dropped |residual| or |bias|, a
signed instead of an absolute product, or a term summed over the wrong taps
fails one of these."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth

CASES = [
    # n, cin, h, w, cout, kh, kw, sh, sw, ph, pw, dh, dw, groups
    (1, 8, 9, 9, 8, 3, 3, 1, 1, 1, 1, 1, 1, 1),
    (2, 4, 7, 10, 6, 3, 3, 2, 2, 1, 1, 1, 1, 1),
    (1, 6, 8, 8, 4, 2, 3, 1, 2, 0, 1, 2, 1, 2),
    (2, 8, 6, 6, 8, 3, 3, 1, 1, 1, 1, 1, 1, 8),      # depthwise
    (1, 3, 15, 15, 5, 7, 7, 2, 2, 3, 3, 1, 1, 1),    # stem-like
    (3, 16, 4, 4, 8, 1, 1, 1, 1, 0, 0, 1, 1, 1),     # pointwise
]


def _abs64(t):
    return t.to(torch.float64).abs()


def _scale_torch(x, w, case, bias, residual):
    n, cin, h, wd, cout, kh, kw, sh, sw, ph, pw, dh, dw, groups = case
    a = F.conv2d(_abs64(x).permute(0, 3, 1, 2), _abs64(w).permute(0, 3, 1, 2),
                 None if bias is None else _abs64(bias), stride=(sh, sw), padding=(ph, pw),
                 dilation=(dh, dw), groups=groups).permute(0, 2, 3, 1)
    if residual is not None:
        a = a + _abs64(residual)
    return a.numpy()


def _draw(case, dt, seed):
    n, cin, h, wd, cout, kh, kw, sh, sw, ph, pw, dh, dw, groups = case
    x = synth.normal((n, h, wd, cin), dt, seed)
    w = synth.normal((cout, kh, kw, cin // groups), dt, seed + 1)
    bias = synth.normal((cout,), dt, seed + 2)
    ho, wo = oracle.out_dim(h, kh, sh, ph, dh), oracle.out_dim(wd, kw, sw, pw, dw)
    res = synth.normal((n, ho, wo, cout), dt, seed + 3)
    return x, w, bias, res


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("with_bias,with_res", [(False, False), (True, False), (False, True),
                                                (True, True)])
def test_conv_scale_is_abs_conv(case, dt, with_bias, with_res):
    seed = 7000 + CASES.index(case) * 40 + ["f32", "bf16", "f16"].index(dt) * 4 + \
        2 * with_bias + with_res
    x, w, bias, res = _draw(case, dt, seed)
    bias = bias if with_bias else None
    res = res if with_res else None
    _, a, _ = oracle.conv2d(x, w, *case, bias=bias, residual=res, act=oracle.ACT_RELU)
    ref = _scale_torch(x, w, case, bias, res)
    # sums of at most a few hundred nonnegative doubles: orders differ by ulps
    assert np.all(np.abs(a - ref) <= 1e-13 * ref), float(np.max(np.abs(a - ref)))


@pytest.mark.parametrize("case", CASES)
def test_sampled_conv_scale_matches(case):
    x, w, bias, res = _draw(case, "bf16", 7500 + CASES.index(case))
    ref = _scale_torch(x, w, case, bias, res).reshape(-1)
    idx = np.unique(np.concatenate([synth.rng(3).integers(0, ref.size, 64), [0, ref.size - 1]]))
    _, a = oracle.conv2d_at(x, w, idx, *case, bias=bias, residual=res, act=oracle.ACT_RELU6)
    assert np.all(np.abs(a - ref[idx]) <= 1e-13 * ref[idx])


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
def test_fc_scale_is_abs_matmul(dt):
    m, k, n = 7, 45, 19
    x = synth.normal((m, k), dt, 7600)
    w = synth.normal((n, k), dt, 7601)
    b = synth.normal((n,), dt, 7602)
    r = synth.normal((m, n), dt, 7603)
    _, a = oracle.fc(x, w, m, k, n, bias=b, residual=r, act=oracle.ACT_RELU)
    ref = (np.abs(x.double().numpy()) @ np.abs(w.double().numpy()).T
           + np.abs(b.double().numpy())[None, :] + np.abs(r.double().numpy()))
    assert np.all(np.abs(a - ref) <= 1e-13 * ref)
    _, a0 = oracle.fc(x, w, m, k, n)
    ref0 = np.abs(x.double().numpy()) @ np.abs(w.double().numpy()).T
    assert np.all(np.abs(a0 - ref0) <= 1e-13 * ref0)


def test_skipping_leaves_scale_unchanged():
    """Skipped terms hold a zero activation, so |x w| of each is 0: the scale
    with a skip mask equals the scale without one (and the torch one)."""
    case = (2, 16, 6, 6, 8, 3, 3, 1, 1, 1, 1, 1, 1, 1)
    x = synth.sparse_nhwc(2, 6, 6, 16, 0.7, "bf16", 7700)
    w = synth.normal((8, 3, 3, 16), "bf16", 7701)
    st = oracle.measure(x.reshape(72, 16), 72, 16, 1, 8)
    _, a_skip, _ = oracle.conv2d(x, w, *case, skip_mask=st["mask"], skip_rows=1, skip_cols=8)
    _, a_dense, _ = oracle.conv2d(x, w, *case)
    assert np.array_equal(a_skip, a_dense)
    ref = _scale_torch(x, w, case, None, None)
    assert np.all(np.abs(a_dense - ref) <= 1e-13 * ref)


def test_scale_bounds_the_value():
    """|y| <= A before any activation (triangle inequality), with equality
    when every term has the same sign."""
    case = (1, 8, 5, 5, 4, 3, 3, 1, 1, 1, 1, 1, 1, 1)
    x, w, bias, res = _draw(case, "f32", 7800)
    y, a, _ = oracle.conv2d(x, w, *case, bias=bias, residual=res)
    assert np.all(np.abs(y) <= a * (1 + 1e-15))
    xp = x.abs()
    wp = w.abs()
    y2, a2, _ = oracle.conv2d(xp, wp, *case, bias=bias.abs(), residual=res.abs())
    assert np.all(np.abs(y2 - a2) <= 1e-13 * a2)
