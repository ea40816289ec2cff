"""Host-side checks of libsparoa.so (no GPU needed): every declared symbol is
exported, the host-only calls (intensity, routing) match the oracle bit for
bit, and argument validation rejects bad calls before any device work."""
import os
import re

import ctypes

import numpy as np
import pytest

import oracle
from paper_2511_19457_amd import abi

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "sparoa.h")


def _declared():
    text = open(HEADER).read()
    decl = r"^(?:sparoa_status|uint32_t|const char)\s+\*?(sparoa_[a-z0-9_]+)\("
    return sorted(set(re.findall(decl, text, flags=re.M)))


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert len(names) >= 20
    for n in names:
        assert hasattr(abi._L, n), f"{n} declared in sparoa.h but not exported"
    assert sorted(abi.EXPORTS) == names


def test_abi_version_and_status_strings():
    assert abi.sparoa_abi_version() == 4
    assert abi.sparoa_status_string(0) == "ok"
    assert abi.sparoa_status_string(3) == "workspace too small"


def _odt(d):
    return {abi.F32: oracle.F32, abi.F16: oracle.F16, abi.BF16: oracle.BF16}[d]


def test_conv_intensity_matches_oracle():
    g = np.random.default_rng(3)
    for _ in range(500):
        groups = int(g.choice([1, 1, 2, 4]))
        args = dict(n=int(g.integers(1, 64)), c_in=groups * int(g.integers(1, 300)),
                    h=int(g.integers(1, 300)), w=int(g.integers(1, 300)),
                    c_out=groups * int(g.integers(1, 300)), kh=int(g.integers(1, 8)),
                    kw=int(g.integers(1, 8)), sh=int(g.integers(1, 4)), sw=int(g.integers(1, 4)),
                    ph=int(g.integers(0, 4)), pw=int(g.integers(0, 4)), dh=int(g.integers(1, 3)),
                    dw=int(g.integers(1, 3)), groups=groups)
        dt = int(g.integers(0, 3))
        hb = int(g.integers(0, 2))
        try:
            ref = oracle.conv_intensity(*args.values(), dt=_odt(dt), has_bias=hb)
        except ValueError:
            with pytest.raises(abi.SparoaError):
                abi.sparoa_op_intensity_conv(abi.conv_desc(**args, dtype=dt, has_bias=hb))
            continue
        got = abi.sparoa_op_intensity_conv(abi.conv_desc(**args, dtype=dt, has_bias=hb))
        assert got == ref


def test_fc_intensity_matches_oracle_and_overflow():
    g = np.random.default_rng(4)
    for _ in range(300):
        m, k, n = (int(v) for v in g.integers(1, 10000, size=3))
        dt = int(g.integers(0, 3))
        assert abi.sparoa_op_intensity_fc(abi.fc_desc(m, k, n, dt)) == \
            oracle.fc_intensity(m, k, n, _odt(dt))
    with pytest.raises(abi.SparoaError) as e:
        abi.sparoa_op_intensity_fc(abi.fc_desc(2**40, 2**20, 2**10))
    assert e.value.status == 1


def test_route_matches_oracle():
    g = np.random.default_rng(5)
    for _ in range(3000):
        numel = int(g.integers(1, 10**9))
        zeros = int(g.integers(0, numel + 1))
        nb = int(g.integers(0, 1000))
        zb = int(g.integers(0, nb + 1)) if nb else 0
        inten = float(g.choice([g.uniform(0, 1000), 315.0, 20.0]))
        s_thr = float(g.choice([g.uniform(0, 1), 0.5, zeros / numel]))
        c_thr = float(g.choice([315.0, 20.0, inten]))
        dw = int(g.integers(0, 2))
        mode = int(g.integers(0, 2))
        ref = oracle.route(zeros, numel, zb, nb, inten, dw, s_thr, c_thr, mode)
        c = dict(zeros=zeros, numel=numel, zero_blocks=zb, num_blocks=nb)
        i = dict(macs=0, flops=0, bytes=0, intensity=inten)
        if ref < 0:
            with pytest.raises(abi.SparoaError):
                abi.sparoa_route(c, i, dw, s_thr, c_thr, mode)
        else:
            assert abi.sparoa_route(c, i, dw, s_thr, c_thr, mode) == ref


def test_route_invalid_inputs():
    c = dict(zeros=1, numel=2, zero_blocks=0, num_blocks=0)
    i = dict(macs=0, flops=0, bytes=0, intensity=1.0)
    for args in ((c, i, 0, float("nan"), 1.0, 1), (c, i, 0, 0.5, 1.0, 0), (c, i, 0, 0.5, 1.0, 9)):
        with pytest.raises(abi.SparoaError) as e:
            abi.sparoa_route(*args)
        assert e.value.status == 1


def test_mask_words():
    assert abi.sparoa_mask_words(64, 4096, 16, 16) == (4 * 256 + 31) // 32
    assert abi.sparoa_mask_words(3, 5, 2, 2) == 1
    with pytest.raises(abi.SparoaError):
        abi.sparoa_mask_words(0, 5, 2, 2)


FAKE = 0x10000   # an aligned address never dereferenced: calls below fail validation first


def test_validation_rejects_before_device_work():
    d = abi.conv_desc(1, 64, 8, 8, 64, 3, 3, 1, 1, 1, 1)
    # null x
    with pytest.raises(abi.SparoaError) as e:
        abi.sparoa_conv2d(d, abi.PATH_DENSE_MFMA, None, FAKE, None, None, 0, None, FAKE)
    assert e.value.status == 1
    # skip path without a mask
    with pytest.raises(abi.SparoaError) as e:
        abi.sparoa_conv2d(d, abi.PATH_SKIP_MFMA, FAKE, FAKE, None, None, 0, None, FAKE)
    assert e.value.status == 1
    # misaligned pointer
    with pytest.raises(abi.SparoaError) as e:
        abi.sparoa_conv2d(d, abi.PATH_DENSE_MFMA, FAKE + 2, FAKE, None, None, 0, None, FAKE)
    assert e.value.status == 2
    # grouped non-depthwise conv
    g2 = abi.conv_desc(1, 64, 8, 8, 64, 3, 3, 1, 1, 1, 1, groups=2)
    with pytest.raises(abi.SparoaError) as e:
        abi.sparoa_conv2d(g2, abi.PATH_DENSE_MFMA, FAKE, FAKE, None, None, 0, None, FAKE)
    assert e.value.status == 2
    # empty output
    with pytest.raises(abi.SparoaError) as e:
        abi.sparoa_op_intensity_conv(abi.conv_desc(1, 4, 2, 2, 4, 5, 5))
    assert e.value.status == 1
    # has_bias without bias
    with pytest.raises(abi.SparoaError) as e:
        abi.sparoa_fc(abi.fc_desc(4, 64, 64, has_bias=1), 0, FAKE, FAKE, None, None, 0, None,
                      FAKE)
    assert e.value.status == 1
    # a BW FC the weight-streaming kernel cannot take (m > 64, or fp32) runs
    # the implicit GEMM on w[n][k], with that kernel's bitmap granularity
    big = abi.fc_desc(65, 64, 64)
    assert abi.sparoa_fc_skip_block(big, abi.PATH_SKIP_BW) == (1, 8)
    assert not abi.sparoa_fc_uses_packed(big, abi.PATH_SKIP_BW)
    small = abi.fc_desc(64, 64, 64)
    assert abi.sparoa_fc_skip_block(small, abi.PATH_SKIP_BW) == (64, 1)
    assert abi.sparoa_fc_uses_packed(small, abi.PATH_DENSE_BW)
    assert not abi.sparoa_fc_uses_packed(small, abi.PATH_DENSE_MFMA)
    assert not abi.sparoa_fc_uses_packed(abi.fc_desc(8, 64, 64, abi.F32), abi.PATH_DENSE_BW)
    # measurement: zero rows, samples not dividing rows, misaligned x
    counts = FAKE
    for args, status in (((FAKE, 0, 8, 0, 0, 0, counts), 1),
                         ((FAKE, 6, 8, 0, 0, 4, counts, None, FAKE), 1),
                         ((FAKE + 8, 6, 8, 0, 0, 0, counts), 2)):
        with pytest.raises(abi.SparoaError) as e:
            abi.sparoa_measure_sparsity(*args, dtype=abi.BF16)
        assert e.value.status == status


def test_workspace_too_small_is_reported():
    # cfg1 conv needs split-K scratch; passing none must fail before launch
    d = abi.conv_desc(1, 64, 56, 56, 64, 3, 3, 1, 1, 1, 1, dtype=abi.F32)
    need = abi.sparoa_conv2d_workspace_size(d, abi.PATH_DENSE_MFMA)
    assert need > 0
    with pytest.raises(abi.SparoaError) as e:
        abi.sparoa_conv2d(d, abi.PATH_DENSE_MFMA, FAKE, FAKE, None, None, 0, None, FAKE)
    assert e.value.status == 3


def test_tiling_and_skip_block_queries():
    d = abi.conv_desc(32, 256, 14, 14, 256, 3, 3, 1, 1, 1, 1)
    assert abi.sparoa_conv2d_skip_block(d, abi.PATH_SKIP_MFMA) == (1, 8)
    tr, kc = abi.sparoa_conv2d_tiling(d, abi.PATH_SKIP_MFMA)
    assert tr in (64, 128, 256) and kc == 64          # channels % 64 == 0: 64-wide chunks
    d24 = abi.conv_desc(2, 24, 14, 14, 144, 1, 1)
    tr, kc = abi.sparoa_conv2d_tiling(d24, abi.PATH_SKIP_MFMA)
    assert tr in (64, 128) and kc == 32               # general kernel: 32-wide chunks
    d32 = abi.conv_desc(1, 64, 56, 56, 64, 3, 3, 1, 1, 1, 1, dtype=abi.F32)
    assert abi.sparoa_conv2d_tiling(d32, abi.PATH_DENSE_MFMA)[1] == 32
    stem = abi.conv_desc(32, 3, 224, 224, 64, 7, 7, 2, 2, 3, 3)   # direct small-channel kernel
    assert abi.sparoa_conv2d_tiling(stem, abi.PATH_SKIP_MFMA) == (16, 32)
    assert abi.sparoa_conv2d_workspace_size(stem, abi.PATH_DENSE_MFMA) == 0
    # its limits: 16-bit, C_in <= 4, C_out in {16, 32, 64}, dilation 1 (else the general kernel)
    for desc in (abi.conv_desc(2, 4, 40, 40, 32, 3, 3, 1, 1, 1, 1),
                 abi.conv_desc(2, 1, 40, 40, 16, 5, 5, 2, 2, 2, 2, dtype=abi.F16)):
        assert abi.sparoa_conv2d_tiling(desc, abi.PATH_DENSE_MFMA) == (16, 32)
    for desc in (abi.conv_desc(2, 5, 40, 40, 32, 3, 3, 1, 1, 1, 1),
                 abi.conv_desc(2, 3, 40, 40, 48, 3, 3, 1, 1, 1, 1),
                 abi.conv_desc(2, 3, 40, 40, 32, 3, 3, 1, 1, 1, 1, dtype=abi.F32),
                 abi.conv_desc(2, 3, 40, 40, 32, 3, 3, 1, 1, 2, 2, 2, 2)):
        assert abi.sparoa_conv2d_tiling(desc, abi.PATH_DENSE_MFMA)[0] != 16
    f = abi.fc_desc(8, 4096, 4096)
    assert abi.sparoa_fc_skip_block(f, abi.PATH_SKIP_BW) == (8, 1)
    assert abi.sparoa_fc_tiling(f, abi.PATH_SKIP_BW) == (8, 1)
    # two layouts of 16-column panels: k-major, then 32-k chunks (k rounded up)
    assert abi.sparoa_fc_packed_bytes(f) == 2 * 4096 * 4096 * 2
    assert abi.sparoa_fc_packed_bytes(abi.fc_desc(1, 100, 65)) == 80 * 100 * 2 + 80 * 128 * 2


def test_reads_mask_queries():
    """Which conv kernels read x's bitmap: the implicit GEMM's skip forms;
    not the dense paths, nor the kernels that test x themselves."""
    c3 = abi.conv_desc(2, 64, 14, 14, 64, 3, 3, 1, 1, 1, 1)
    assert abi.sparoa_conv2d_reads_mask(c3, abi.PATH_SKIP_MFMA)
    assert not abi.sparoa_conv2d_reads_mask(c3, abi.PATH_DENSE_MFMA)
    pw = abi.conv_desc(11, 64, 56, 56, 96, 1, 1)         # the pointwise kernel on the BW path
    assert abi.sparoa_conv2d_tiling(pw, abi.PATH_SKIP_BW) == (16, 32)
    assert not abi.sparoa_conv2d_reads_mask(pw, abi.PATH_SKIP_BW)
    assert abi.sparoa_conv2d_reads_mask(pw, abi.PATH_SKIP_MFMA)
    dw = abi.conv_desc(2, 32, 16, 16, 32, 3, 3, 1, 1, 1, 1, groups=32)
    assert not abi.sparoa_conv2d_reads_mask(dw, abi.PATH_SKIP_BW)
    stem = abi.conv_desc(32, 3, 224, 224, 64, 7, 7, 2, 2, 3, 3)
    assert not abi.sparoa_conv2d_reads_mask(stem, abi.PATH_SKIP_MFMA)
    # the routed form: the family the intensity threshold selects
    inten = abi.sparoa_op_intensity_conv(pw)["intensity"]
    assert not abi.sparoa_conv2d_routed_reads_mask(pw, 0.5, inten * 2, abi.ROUTE_BLOCK)
    assert abi.sparoa_conv2d_routed_reads_mask(pw, 0.5, 0.0, abi.ROUTE_BLOCK)
    assert not abi.sparoa_conv2d_routed_reads_mask(dw, 0.5, 0.0, abi.ROUTE_BLOCK)


@pytest.mark.skipif(os.path.exists("/dev/kfd"),
                    reason="host-only check: the fake device pointers must never reach a GPU")
def test_counts_only_and_null_mask_validation():
    """Rejected before any device work: a counts-only output measurement with
    cols % 8 != 0, y_mask without y_counts, and a null x bitmap for a routed
    conv whose skip kernel reads one."""
    c3 = abi.conv_desc(2, 64, 14, 14, 64, 3, 3, 1, 1, 1, 1)
    for desc, y_counts, y_mask in ((abi.conv_desc(2, 64, 14, 14, 60, 3, 3, 1, 1, 1, 1,
                                                  dtype=abi.F32), FAKE, None),
                                   (abi.conv_desc(2, 64, 14, 14, 60, 3, 3, 1, 1, 1, 1), FAKE,
                                    None),
                                   (c3, None, FAKE)):
        with pytest.raises(abi.SparoaError) as e:
            abi.sparoa_conv2d_routed_measured(desc, 0.5, 0.0, abi.ROUTE_BLOCK, FAKE, FAKE, FAKE,
                                              None, None, 0, FAKE, FAKE, y_counts, y_mask, None)
        assert e.value.status == 1
    with pytest.raises(abi.SparoaError) as e:
        abi.sparoa_conv2d_routed(c3, 0.5, 0.0, abi.ROUTE_BLOCK, FAKE, FAKE, FAKE, None, None, 0,
                                 None, FAKE)
    assert e.value.status == 1
    with pytest.raises(abi.SparoaError) as e:
        abi.sparoa_fc_routed_measured(abi.fc_desc(64, 256, 100), 0.5, 0.0, abi.ROUTE_BLOCK, FAKE,
                                      FAKE, FAKE, None, None, None, 0, FAKE, FAKE, FAKE, None)
    assert e.value.status == 1


@pytest.mark.skipif(os.path.exists("/dev/kfd"),
                    reason="host-only check: the fake device pointers must never reach a GPU")
def test_executor_chained_batch_without_events_fails_cleanly_without_a_gpu():
    """Regression: a chained batch (op 1 reads op 0's output) with no events
    takes the op-by-op route; with no GPU present it must report the HIP
    error of its first launch, not dereference the missing event array."""
    d = abi.fc_desc(128, 256, 256, abi.BF16)
    y0 = 0x200000000
    t = abi.Thresholds(0.5, 315.0, abi.ROUTE_BLOCK)
    ops = [abi.FcOp(d, 0x100000000, 0x110000000, 0x120000000, None, None, abi.ACT_RELU,
                    0x130000000, 0x140000000, y0, 0x150000000, 1 << 20, 0x160000000, t),
           abi.FcOp(d, y0, 0x170000000, 0x180000000, None, None, abi.ACT_RELU, 0x190000000,
                    0x1a0000000, 0x1b0000000, 0x1c0000000, 1 << 20, 0x1d0000000, t)]
    arr = (abi.FcOp * 2)(*ops)
    st = abi._L.sparoa_fc_ops_run(arr, 2, None, None, None)
    assert st == 4, abi._L.sparoa_last_error()


def _fake_op(d, base, t, ws_bytes=1 << 26, w_nk=True):
    """An FC op whose device pointers are distinct fake addresses."""
    a = [base + (i << 28) for i in range(9)]
    return abi.FcOp(d, a[0], a[1] if w_nk else None, a[2], None, None, abi.ACT_RELU, a[3], a[4],
                    a[5], a[6], ws_bytes, a[7], t)


@pytest.mark.skipif(os.path.exists("/dev/kfd"),
                    reason="host-only check: the fake device pointers must never reach a GPU")
@pytest.mark.parametrize("bad", ["workspace", "w_nk"])
def test_executor_validates_every_op_before_any_launch(bad):
    """A batch whose second op fails validation launches nothing: the call
    reports that op's validation error (with no GPU present, any launch
    before it would have reported a HIP error instead)."""
    d = abi.fc_desc(64, 4096, 4096, abi.BF16)
    t = abi.Thresholds(0.5, 0.0, abi.ROUTE_BLOCK)            # MFMA family: split-K workspace
    need = abi.sparoa_fc_workspace_size(d, abi.PATH_SKIP_MFMA)
    assert need > 0
    op1 = _fake_op(d, 0x2000000000, t, ws_bytes=need - 16) if bad == "workspace" else \
        _fake_op(d, 0x2000000000, t, w_nk=False)
    arr = (abi.FcOp * 2)(_fake_op(d, 0x1000000000, t), op1)
    st = abi._L.sparoa_fc_ops_run(arr, 2, None, None, None)
    assert st == (3 if bad == "workspace" else 1), abi._L.sparoa_last_error()
    assert b"op 1" in abi._L.sparoa_last_error()


@pytest.mark.skipif(os.path.exists("/dev/kfd"),
                    reason="host-only check: the fake device pointers must never reach a GPU")
def test_measured_fc_validates_before_measuring():
    """sparoa_fc_measured checks the routed FC's workspace before it launches
    the measurement of x."""
    d = abi.fc_desc(64, 4096, 4096, abi.BF16)
    need = abi.sparoa_fc_workspace_size(d, abi.PATH_SKIP_MFMA)
    with pytest.raises(abi.SparoaError) as e:
        abi._check(abi._L.sparoa_fc_measured(
            ctypes.byref(d), ctypes.byref(abi.Thresholds(0.5, 0.0, abi.ROUTE_BLOCK)),
            0x1000000000, 0x1100000000, None, None, None, abi.ACT_NONE, 0x1200000000,
            0x1300000000, 0x1400000000, 0x1500000000, need - 16, None, None))
    assert e.value.status == 3
